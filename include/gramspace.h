/*
 * gramspace.h -- C ABI of the Gram-Space operator library for MI355X (gfx950).
 *
 * Gram-Space (Wang & Li, "Gram-Space: Structure-Preserving Codebook
 * Compression for Memory-Efficient Neuro-Symbolic AI") factors a VSA codebook
 * into an orthonormal basis and per-vector coordinates ("Gram-loc"), runs the
 * matrix-space operators (probability vectorisation, similarity, attention
 * score) on the coordinates, and restores vectors to the original domain only
 * before component-wise operators such as binding.
 *
 * Notation.  The paper stores the codebook as W (D x M, one codebook vector
 * per column), the basis as U (D x k) and the Gram-loc codebook as
 * T = U^T W (Sec. 3.1, Eq. 1).  This library stores the transposes, row-major:
 *   C  (M x D)  codebook, row j = codebook vector c_j       (= W^T)
 *   Q  (r x D)  orthonormal basis, row k = basis vector q_k (= U^T)
 *   R  (M x r)  Gram-loc of the codebook, C = R Q           (= T^T)
 *   T  (B x r)  Gram-loc of a batch of B vectors, x_b = T_b Q
 * r is the algebraic rank of C (Sec. 3.2).  All matrices are row-major with a
 * leading dimension (elements between consecutive rows) ld >= columns.
 *
 * Row padding.  When both bf16 operands of a contraction have 16-byte aligned
 * rows (base address 16-byte aligned and ld a multiple of 8), rows are read
 * in 16-byte units, up to column ceil(columns / 8) * 8 - 1 <= ld - 1: the
 * row's padding may be read but never contributes (it may hold anything,
 * NaN included).  Such operands take the asynchronous-load paths; any other
 * layout is accepted as well.
 *
 * Memory and ownership.  Every matrix argument is a device pointer (HIP
 * device memory of the current device) unless marked HOST.  The caller
 * allocates every buffer, including workspace; the library allocates no
 * device memory and never frees caller memory (the one exception is the
 * static scratch array of gs_compress_noalloc, part of the loaded code
 * object).  Besides a thread-local error message it keeps three process-wide
 * caches: whether a HIP device exists, which of its kernels have had their
 * LDS limit raised, and the device address of each GPU's scratch array.  Inputs are
 * read-only.  Outputs must not overlap inputs or each other (GS_ERR_ARG).
 *
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = null stream).
 * Every call except gs_compress only enqueues work on that stream and returns
 * without waiting.  gs_compress synchronises the stream before returning
 * because the rank is returned in host memory.  The allocating compress
 * calls (gs_compress, gs_compress_partitioned, gs_compress_padded) also run
 * part of their work on a second stream of the library's (one per GPU,
 * non-blocking, default priority, created on the first such call on that
 * GPU and kept until the process ends), forked from and joined back into
 * `stream` by events within the call; gs_compress_noalloc runs everything on
 * `stream` and gives the same results bit for bit.
 *
 * Element types.  GS_F32 and GS_BF16 (bfloat16 storage, fp32 arithmetic) for
 * batch data and coordinates; GS_F64 additionally for compress input/outputs.
 * Within one call, the two operands of a contraction have the same type.
 * Scores and attention weights are always fp32.  Conversions to bf16 round to
 * nearest even.
 *
 * Errors.  Every call returns a gs_status; gs_last_error() returns a text
 * description of the last failure on the calling thread.  Arguments are
 * validated before any device work; on a validation failure nothing is
 * written.  A zero batch (B == 0) is valid and does nothing; its batch-sized
 * buffers may then be NULL.  A failing launch
 * returns GS_ERR_DEVICE and leaves outputs undefined.
 *
 * Environment.  GS_DEBUG (any value): every call waits for the device after
 * its launches and reports a failure found there as GS_ERR_DEVICE (slow; for
 * locating a failing call).  GS_LOG (any value but "0"): one line on stderr
 * per rejected call (status and message) and per launched call.
 */
#ifndef GRAMSPACE_H
#define GRAMSPACE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GS_ABI_VERSION 2

typedef enum {
    GS_OK = 0,
    GS_ERR_ARG = 1,        /* null pointer, bad enum, negative size, overlap */
    GS_ERR_SHAPE = 2,      /* inconsistent sizes or leading dimensions       */
    GS_ERR_DTYPE = 3,      /* unsupported element-type combination          */
    GS_ERR_ALIGN = 4,      /* pointer not aligned to its element size        */
    GS_ERR_WORKSPACE = 5,  /* workspace missing or too small                 */
    GS_ERR_NUMERIC = 6,    /* non-finite codebook entry                      */
    GS_ERR_DEVICE = 7      /* no usable GPU, or a HIP call failed            */
} gs_status;

typedef enum { GS_F32 = 0, GS_BF16 = 1, GS_F64 = 2 } gs_dtype;

/* Similarity function of Sec. 2.2: a scaled dot product, or the dot product
   of the normalised vectors (cosine). */
typedef enum { GS_SIM_DOT = 0, GS_SIM_COSINE = 1 } gs_sim_mode;

/*
 * Structure flag for the codebook coordinates R of gs_prob2vec, gs_similarity
 * and gs_attention: OR it into rt when R is lower echelon, R[j][k] == 0 for
 * every k > j.  gs_compress returns R in this form: its basis is built from
 * the codebook vectors in index order, so c_j lies in the span of the first
 * j + 1 basis vectors (Eq. 1).  The large products then skip the blocks of R
 * above its diagonal (at r = M about half the work of P R, T R^T and A R);
 * for finite P, T and A the results are those of the same call without the
 * flag.  Entries of R above the diagonal may then go unread: if they are not
 * zero, the results are undefined.  Cosine scores whose ||x_b|| comes from T
 * (qnorm2 == NULL) keep the full range.
 */
#define GS_ECHELON 0x100

/* Component-wise operator applied after restoring two vectors. */
typedef enum { GS_BIND_NONE = 0, GS_BIND_MUL = 1 } gs_bind;

/* Component-wise binding operator of gs_bind_restored. */
typedef enum { GS_BINDOP_MUL = 0, GS_BINDOP_XOR = 1, GS_BINDOP_CONV = 2, GS_BINDOP_CORR = 3 } gs_bind_op;

/* ABI version of the loaded library (GS_ABI_VERSION of its build). */
int gs_abi_version(void);

/* Text of the last error on the calling thread ("" if none).  The pointer
   stays valid until the next gs_* call on the same thread. */
const char *gs_last_error(void);

/*
 * gs_compress_workspace -- bytes of device workspace gs_compress needs for an
 * M x D codebook.  Returns 0 for invalid sizes.
 */
size_t gs_compress_workspace(int64_t M, int64_t D);

/*
 * gs_compress -- Gram-Space compression (Sec. 3.1 Eq. 1; rank Sec. 3.2;
 * construction at initialisation Sec. 3.3).
 *
 * Builds an orthonormal basis Q of the row space of the codebook C and its
 * coordinates R with C = R Q, by block Gram-Schmidt with re-orthogonalisation
 * over panels of codebook rows, in fp64 (the rows of a panel are
 * orthogonalised among themselves in the space of the panel's triangular
 * factor, by modified Gram-Schmidt with a second projection wherever the
 * first took away most of a row's norm).  Codebook rows are taken in index
 * order; row i is dependent (adds no basis vector) when the norm of its part
 * outside the current span is <= tol * ||c_i||.  Kept rows
 * are listed in `kept`, so basis vector k comes from codebook row kept[k].  R
 * is lower-echelon: R[i, k] = <c_i, q_k> for basis vectors created before row
 * i, R[kept[k], k] > 0, zero elsewhere.  With these rules Q and R are unique.
 *
 *   C      in   M x D, ct in {F32, BF16, F64}, leading dimension ldc >= D
 *   M, D        1 <= M <= D (D < M: gs_compress_partitioned)
 *   tol         relative rank threshold, 0 <= tol < 1 (1e-10 recommended)
 *   Q      out  rank x D, qt in {F64, F32, BF16}, ldq >= D; rows rank..M-1
 *               are zero-filled (capacity M rows)
 *   R      out  M x rank, rt in {F64, F32, BF16}, ldr >= M; columns rank..M-1
 *               are zero-filled (capacity M columns)
 *   kept   out  int32[M] device, nullable; entries rank..M-1 set to -1
 *   cnorm  out  float[M] device, nullable: ||c_i|| (used by cosine similarity)
 *   rank   out  HOST int32
 *   ws          device workspace of >= gs_compress_workspace(M, D) bytes,
 *               256-byte aligned; contents on return are unspecified
 *   stream      synchronised before return (part of the work runs on the
 *               library's second stream, joined back before return)
 * Errors: GS_ERR_NUMERIC if C holds a NaN or infinity (detected on the device;
 * outputs are then undefined), or if the re-orthonormalisation of a panel
 * meets a Gram matrix that is not positive definite (not expected for finite
 * input).
 */
gs_status gs_compress(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc,
                      double tol,
                      void *Q, gs_dtype qt, int64_t ldq,
                      void *R, gs_dtype rt, int64_t ldr,
                      int32_t *kept, float *cnorm, int32_t *rank,
                      void *ws, size_t ws_bytes, void *stream);

/*
 * gs_compress_padded -- a basis of k > M vectors (Sec. 3.1: k may exceed M
 * to preserve representation sparsity, the orthonormal basis being augmented
 * by zero-padding and a linear transformation that spreads the signal over
 * the added dimensions).  The basis of the codebook (as gs_compress builds
 * it, rank r) is completed to k orthonormal vectors by the unit vectors
 * e_0, e_1, ... taken in index order, each kept only if it leaves the span
 * built so far by more than tol (the codebook's coordinates on the added
 * vectors are zero: its coordinates are zero-padded).  With H given, an
 * orthogonal k x k matrix (fp64, device, row-major, leading dimension ldh),
 * the basis and the coordinates are transformed together:
 *   Q = H Q_k    (k x D, orthonormal rows)       R = R_k H^T    (M x k)
 * so C = R Q, every inner product and norm of coordinates is unchanged, and
 * reconstruction x = t Q is exact; H = NULL means the identity (plain zero
 * padding).  H must be orthogonal for these properties (not checked); a
 * normalised Hadamard matrix spreads each coordinate vector's energy evenly
 * over the k dimensions.
 *   M, D, k     M <= k and M + k <= D
 *   Q      out  k x D, qt in {F64, F32, BF16}, ldq >= D
 *   R      out  M x k, rt in {F64, F32, BF16}, ldr >= k
 *   kept   out  int32[M] device, nullable: the codebook rows that made the
 *               first r basis vectors (before the transformation), -1 after
 *   cnorm  out  float[M] device, nullable
 *   rank   out  HOST int32: r, the codebook's rank
 *   ws          device workspace of >= gs_compress_padded_workspace(M, D, k)
 *               bytes, 256-byte aligned
 * Errors as gs_compress.
 */
size_t gs_compress_padded_workspace(int64_t M, int64_t D, int64_t k);

gs_status gs_compress_padded(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc,
                             double tol, int64_t k, const double *H, int64_t ldh,
                             void *Q, gs_dtype qt, int64_t ldq,
                             void *R, gs_dtype rt, int64_t ldr,
                             int32_t *kept, float *cnorm, int32_t *rank,
                             void *ws, size_t ws_bytes, void *stream);

/*
 * gs_compress_partitioned -- compression of a codebook with more entries than
 * dimensions (Sec. 3.1: when D < M the entries are split into subsets of at
 * most D, each with its own orthonormal basis, the subsets put side by side
 * again after reconstruction).  Rows are taken in consecutive subsets of
 * `subset` rows (1 <= subset <= D; the last one may be shorter); each is
 * compressed as by gs_compress.  With subset ranks r_g and offsets
 * o_g = r_0 + ... + r_{g-1}:
 *   Q      out  the subsets' bases stacked: rows o_g .. o_g + r_g - 1 are the
 *               basis of subset g (orthonormal within a subset, not across
 *               subsets); capacity M x D, rows past the total rank zero
 *   R      out  block diagonal: the rows of subset g hold their coordinates
 *               in columns o_g .. o_g + r_g - 1, zero elsewhere; capacity
 *               M x M (ldr >= M); C = R Q, and R is lower echelon
 *   kept   out  int32[M] device, nullable: codebook row of each basis vector,
 *               -1 past the total rank
 *   cnorm  out  float[M] device, nullable
 *   ranks  out  HOST int32[ceil(M / subset)]: r_g
 *   rank   out  HOST int32: the total, sum of r_g (the rows of Q in use)
 *   ws          workspace of >= gs_compress_workspace(min(subset, M), D) bytes
 * Any M >= 1 is accepted (subset = M <= D is gs_compress).  With these
 * outputs: gs_project(X, Q) gives each subset's coordinates of x side by side,
 * and gs_similarity of them against R (dot, or cosine with the dense ||x||^2
 * from gs_project and cnorm) is exactly the similarity with every codebook
 * entry; gs_prob2vec(P, R) gives coefficients whose gs_reconstruct against Q
 * is p C.  Those coefficients are not the projection of p C (the stacked
 * basis is not orthonormal), so they are restored, not compared directly.
 */
gs_status gs_compress_partitioned(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc,
                                  double tol, int64_t subset,
                                  void *Q, gs_dtype qt, int64_t ldq,
                                  void *R, gs_dtype rt, int64_t ldr,
                                  int32_t *kept, float *cnorm, int32_t *ranks, int32_t *rank,
                                  void *ws, size_t ws_bytes, void *stream);

/*
 * gs_compress_noalloc -- gs_compress for callers that cannot allocate device
 * memory (code under stream capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation and arguments without the
 * workspace, which comes instead from a static array of
 * GS_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * (from the first call on that device until the process ends).  The call
 * allocates nothing and creates no stream or event: its work runs on `stream`
 * alone.  Codebooks whose workspace, gs_compress_workspace(M, D),
 * exceeds the array are rejected with GS_ERR_WORKSPACE (64 MiB: e.g. up to
 * 1000 x 4096 or 256 x 8192 in fp64 working precision).  All calls on one GPU
 * share its array: calls that overlap in time on the same GPU (other threads,
 * other streams) race and give undefined results; each call initialises what
 * it needs, so consecutive calls are independent.  The scratch memory is the
 * current device's.
 */
#define GS_NOALLOC_SCRATCH_BYTES (64u << 20)

gs_status gs_compress_noalloc(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc,
                              double tol,
                              void *Q, gs_dtype qt, int64_t ldq,
                              void *R, gs_dtype rt, int64_t ldr,
                              int32_t *kept, float *cnorm, int32_t *rank, void *stream);

/*
 * gs_project -- Gram-loc of a batch (Sec. 3.1: t = U^T x):  T = X Q^T.
 *
 *   X      in   B x D, xt in {F32, BF16}, ldx >= D
 *   Q      in   r x D, qt == xt, ldq >= D
 *   T      out  B x r, tt in {F32, BF16}, ldt >= r
 *   xnorm2 out  float[B], nullable: ||x_b||^2 of the dense input, computed in
 *               the same pass (needed for cosine similarity of vectors that
 *               are not in the span of the codebook)
 * fp32 accumulation.
 */
gs_status gs_project(const void *X, gs_dtype xt, int64_t B, int64_t D, int64_t ldx,
                     const void *Q, gs_dtype qt, int64_t r, int64_t ldq,
                     void *T, gs_dtype tt, int64_t ldt,
                     float *xnorm2, void *stream);

/*
 * gs_prob2vec -- probability vectorisation on Gram-loc (Sec. 2.2, Sec. 3.1):
 * the dense v_b = sum_j P[b, j] c_j is never formed; its Gram-loc is
 * T = P R.
 *
 *   P      in   B x M, pt in {F32, BF16}, ldp >= M
 *   R      in   M x r, rt == pt (| GS_ECHELON), ldr >= r (r may exceed M for
 *               a padded basis, gs_compress_padded)
 *   T      out  B x r, tt in {F32, BF16}, ldt >= r
 * fp32 accumulation.
 */
gs_status gs_prob2vec(const void *P, gs_dtype pt, int64_t B, int64_t M, int64_t ldp,
                      const void *R, gs_dtype rt, int64_t r, int64_t ldr,
                      void *T, gs_dtype tt, int64_t ldt, void *stream);

/*
 * gs_prob2vec_sparse -- probability vectorisation (Sec. 2.2, Sec. 3.1) of
 * sparse probability rows: t_b = sum over the stored entries (j, p) of row b
 * of p R_j, the Gram-loc of sum_j p_j c_j, reading only the rows of R the
 * entries name.  Rows come in compressed sparse row form:
 *
 *   rowptr in   int64[B + 1] device: the entries of row b are
 *               rowptr[b] .. rowptr[b + 1] - 1 (rowptr[0] = 0, nondecreasing,
 *               rowptr[B] = nnz)
 *   cols   in   int32[nnz] device: codebook index j of each entry, 0 <= j < M
 *   vals   in   nnz probabilities p, type vt in {F32, BF16}
 *   R      in   M x r, rt == vt (a GS_ECHELON flag is ignored), ldr >= r
 *               (r may exceed M, as for gs_prob2vec with a padded basis)
 *   T      out  B x r, tt in {F32, BF16}, ldt >= r
 * A row's entries are summed in their stored order in fp32; a row without
 * entries gives t = 0.  Entries whose index lies outside [0, M), and pointer
 * ranges outside [0, nnz], are skipped on the device (never read out of
 * bounds); the result is then that of the remaining entries.
 */
gs_status gs_prob2vec_sparse(const int64_t *rowptr, const int32_t *cols, const void *vals, gs_dtype vt,
                             int64_t B, int64_t M, int64_t nnz,
                             const void *R, gs_dtype rt, int64_t r, int64_t ldr,
                             void *T, gs_dtype tt, int64_t ldt, void *stream);

/*
 * gs_similarity -- similarity of each batch vector with every codebook vector,
 * on Gram-loc (Sec. 2.2; invariance Sec. 3.2 Eq. 2-3):
 *   DOT:     S[b, j] = scale * <t_b, R_j>                       (= <x_b, c_j>)
 *   COSINE:  S[b, j] = scale * <t_b, R_j> / (||x_b|| ||c_j||), 0 if a norm is 0
 * with ||x_b||^2 = qnorm2[b] when given (e.g. from gs_project), else ||t_b||^2
 * (exact for vectors in the span, such as prob2vec outputs), and
 * ||c_j|| = cnorm[j] when given, else ||R_j||.
 *
 *   T      in   B x r, tt in {F32, BF16}, ldt >= r
 *   R      in   M x r, rt == tt (| GS_ECHELON), ldr >= r
 *               (r >= 1 and may exceed M: the same call on D-space vectors
 *               and the uncompressed codebook, r = D, is the dense lookup)
 *   qnorm2 in   float[B], nullable;  cnorm in float[M], nullable
 *   S      out  float B x M, nullable, lds >= M
 *   argmax out  int32[B], nullable: index of the largest S[b, :], the lowest
 *               index on an exact tie
 * At least one of S and argmax must be given.  fp32 accumulation.
 */
gs_status gs_similarity(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                        const void *R, gs_dtype rt, int64_t M, int64_t ldr,
                        const float *qnorm2, const float *cnorm,
                        gs_sim_mode mode, float scale,
                        float *S, int64_t lds, int32_t *argmax, void *stream);

/*
 * gs_attention -- attention score over the codebook (Sec. 2.2): the softmax
 * over j of beta * S[b, j], with S as in gs_similarity (same T, R, qnorm2,
 * cnorm, mode and scale), and optionally the attention-weighted sum of the
 * codebook vectors in Gram-loc, O = A R (its dense form is sum_j A[b,j] c_j).
 *
 *   A      out  float B x M, lda >= M (required)
 *   O      out  B x r, ot in {F32, BF16}, ldo >= r, nullable
 */
gs_status gs_attention(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                       const void *R, gs_dtype rt, int64_t M, int64_t ldr,
                       const float *qnorm2, const float *cnorm,
                       gs_sim_mode mode, float scale, float beta,
                       float *A, int64_t lda,
                       void *O, gs_dtype ot, int64_t ldo, void *stream);

/*
 * gs_similarity_attention -- the similarity lookup and the attention weights
 * of one batch from a single evaluation of the scores (Sec. 2.2: the
 * attention score is the softmax of beta times the similarity):
 *   S[b, j]    as gs_similarity computes it (same T, R, qnorm2, cnorm, mode,
 *              scale and conditions)
 *   argmax[b]  the lowest index of the largest S[b, :]
 *   A[b, j]    softmax over j of beta * S[b, j], taken from the fp32 scores
 *              (max-subtracted; any sign of beta)
 *
 *   S      out  float B x M, nullable, lds >= M
 *   argmax out  int32[B], nullable
 *   A      out  float B x M, nullable, lda >= M; when S is NULL the scores
 *               are formed in A and replaced there by the weights
 * At least one of S, argmax and A must be given; the outputs must not
 * overlap each other or the inputs.  Calling gs_similarity and gs_attention
 * gives the same results up to rounding, at about twice the arithmetic.
 */
gs_status gs_similarity_attention(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                                  const void *R, gs_dtype rt, int64_t M, int64_t ldr,
                                  const float *qnorm2, const float *cnorm,
                                  gs_sim_mode mode, float scale,
                                  float *S, int64_t lds, int32_t *argmax,
                                  float beta, float *A, int64_t lda, void *stream);

/*
 * gs_reconstruct -- restore vectors to the original domain (Sec. 3.1 and
 * Sec. 3.3, the "decompose" step): X = T Q.  With bind == GS_BIND_MUL and a
 * second coordinate batch T2, the two restored vectors are bound
 * component-wise (Sec. 2.2; Table 1 "element-wise product") in the same pass:
 * X = (T Q) .* (T2 Q).
 *
 *   T      in   B x r, tt in {F32, BF16}, ldt >= r
 *   T2     in   B x r, same type as T, ldt2 >= r; required iff bind == MUL
 *   Q      in   r x D, qt == tt, ldq >= D
 *   X      out  B x D, xt in {F32, BF16}, ldx >= D
 * fp32 accumulation.
 */
gs_status gs_reconstruct(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                         const void *T2, int64_t ldt2, gs_bind bind,
                         const void *Q, gs_dtype qt, int64_t D, int64_t ldq,
                         void *X, gs_dtype xt, int64_t ldx, void *stream);

/*
 * gs_bind_coords -- binding of two coordinate batches through the original
 * domain in one pass (Sec. 3.3: a component-wise operator runs after the
 * restore and its result is projected back; Sec. 2.2 and Table 1:
 * element-wise product):  Z = ((T Q) .* (T2 Q)) Q^T,  row by row
 *   z_b = ((t_b Q) .* (t2_b Q)) Q^T.
 * The restored and bound vectors stay on the chip: the call equals
 * gs_reconstruct(T, Q, T2, GS_BIND_MUL) followed by gs_project of its result
 * against Q, without the B x D intermediate.
 *
 *   T, T2  in   B x r, f32, ldt, ldt2 >= r; 1 <= r <= 256
 *   Q      in   r x D, f32, ldq >= D
 *   Z      out  B x r, f32, ldz >= r; overlaps none of the inputs
 * fp32 accumulation; each sum over D runs in order over chunks of 32
 * columns.  tt, qt and zt must be GS_F32 (GS_ERR_DTYPE otherwise); r above
 * 256 gives GS_ERR_SHAPE (use the two calls).  The pass saves the B x D
 * write and read of the two calls but holds 128 rows per work-group: it is
 * the faster form for r up to 128 on batches that fill the GPU (at least
 * 256 x 128 rows); at r = 256 the two calls run faster.
 */
gs_status gs_bind_coords(const void *T, gs_dtype tt, int64_t B, int64_t r, int64_t ldt,
                         const void *T2, int64_t ldt2, const void *Q, gs_dtype qt, int64_t D, int64_t ldq,
                         void *Z, gs_dtype zt, int64_t ldz, void *stream);

/*
 * gs_bind_restored -- binding and unbinding of restored vectors, row by row (Sec. 2.2:
 * the modulo-style component-wise operators run in the original domain,
 * after gs_reconstruct; Sec. 3.3: circular convolution).  For each row b:
 *   GS_BINDOP_MUL   Z = X .* Y                        element-wise product
 *   GS_BINDOP_XOR   Z = (X >= 0.5) xor (Y >= 0.5)     binary vectors, 0 / 1
 *   GS_BINDOP_CONV  blockwise circular convolution over consecutive blocks
 *                   of L values: Z[i] = sum_j X[j] Y[(i - j) mod L]  (bind)
 *   GS_BINDOP_CORR  blockwise circular correlation:
 *                   Z[i] = sum_j X[j] Y[(j - i) mod L]  (unbind by Y)
 *
 *   X, Y   in   B x D, type xt in {F32, BF16}, ldx, ldy >= D
 *   L           CONV / CORR block length: a power of two with 2 <= L <= 8192
 *               that divides D (L = D: the whole row); ignored otherwise
 *   Z      out  B x D, type zt in {F32, BF16}, ldz >= D; overlaps neither X
 *               nor Y
 * CONV and CORR go through an fp32 FFT of each block, so each result carries
 * an error of a few fp32 units of log2(L) ||x_block|| ||y_block||.
 */
gs_status gs_bind_restored(const void *X, gs_dtype xt, int64_t B, int64_t D, int64_t ldx,
                           const void *Y, int64_t ldy, gs_bind_op op, int64_t L,
                           void *Z, gs_dtype zt, int64_t ldz, void *stream);

/*
 * gs_soft_select -- the soft-selection pass (Sec. 3.1: probabilities are
 * turned into superposed vectors, which are then compared through attention
 * scores; operators of Sec. 2.2) fused into one launch over up to eight small
 * codebooks.  For every probability row p of group g:
 *   t = p R_g                        (probability vectorisation on Gram-loc)
 *   S[b, j] = scale * sim(t, R_g[j]) (DOT, or COSINE with ||x|| = ||t||: the
 *                                     superposed vector lies in the span of
 *                                     the codebook, Sec. 3.2)
 *   argmax[b] = lowest index of the row maximum of S
 *   A[b, j] = softmax over j of beta * S[b, j]
 * It computes what gs_prob2vec, gs_similarity and gs_attention compute on the
 * same inputs, without storing and re-reading the coordinates in between.
 * `form` chooses how the scores are formed:
 *   GS_SOFT_COORDS  t = p R_g per row, in registers; stored only where T is
 *                   given; scores <t, R_g[j]> from it
 *   GS_SOFT_GRAM    the coordinates are not formed at all: the scores are
 *                   taken through the Gram matrix G = R_g R_g^T (= C C^T,
 *                   Sec. 3.2) of the codebook, <t, R_g[j]> = sum_k p_k G[k][j]
 *                   and ||t||^2 = sum_j p_j <t, R_g[j]>, which equal the
 *                   definitions above up to rounding order; every T must be
 *                   null (GS_ERR_ARG otherwise)
 *   GS_SOFT_AUTO    GS_SOFT_COORDS if some group asks for T, else GS_SOFT_GRAM
 *
 *   groups     HOST array of ngroups descriptors, 1 <= ngroups <= 8; in each,
 *              1 <= r <= M <= 32, B >= 0, and
 *     P        in   B x M probabilities, type pt (F32 or BF16), ldp >= M
 *     R        in   M x r Gram-loc codebook, type pt, ldr >= r
 *     cnorm    in   float[M] codebook norms (cosine), nullable: ||R_j||
 *     T        out  B x r coordinates of the superposed vectors, type tt,
 *                   ldt >= r, nullable
 *     S        out  float B x M scores, lds >= M, nullable
 *     argmax   out  int32[B], nullable
 *     A        out  float B x M attention weights, lda >= M, nullable
 *   Outputs of all groups must overlap neither each other nor any input.
 */
typedef struct {
    const void *P; int64_t ldp;
    const void *R; int64_t ldr;
    const float *cnorm;
    int64_t B, M, r;
    void *T; int64_t ldt;
    float *S; int64_t lds;
    int32_t *argmax;
    float *A; int64_t lda;
} gs_soft_group;

typedef enum { GS_SOFT_AUTO = 0, GS_SOFT_GRAM = 1, GS_SOFT_COORDS = 2 } gs_soft_form;

gs_status gs_soft_select(const gs_soft_group *groups, int ngroups, gs_dtype pt, gs_dtype tt,
                         gs_sim_mode mode, float scale, float beta, gs_soft_form form,
                         void *stream);

#ifdef __cplusplus
}
#endif

#endif /* GRAMSPACE_H */
