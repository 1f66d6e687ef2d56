/*
 * bigcn.h -- C ABI of the MI355X (gfx950) binarized-GCN inference library.
 *
 * The library computes the inference path of Bi-GCN ("Bi-GCN: Binary Graph
 * Convolutional Network", Wang et al., CVPR 2021, Sec. 4.1): each layer
 * binarises its input node features and its weights by sign with
 * full-precision per-bucket scales, multiplies the packed signs with an
 * XNOR / bit-count binary GEMM, and aggregates the rescaled result over the
 * graph with the normalised adjacency.
 *
 * Conventions shared by every entry point
 *  - All pointers except `layers` (bigcn_forward) are DEVICE pointers owned by
 *    the caller; the library never allocates, frees or keeps them.  Inputs
 *    are never written.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Every
 *    call only enqueues work on `stream` and returns; results are ready once
 *    the caller synchronises that stream.  No call synchronises the device.
 *  - Matrices are row-major with a leading dimension (ld*) counted in
 *    elements.  Packed sign rows are arrays of uint64_t words: element k of a
 *    row is bit (k % 64) of word (k / 64), a set bit means +1 (the sign of a
 *    value y is +1 iff y >= 0, so +0 and -0 give +1), and bits at positions
 *    k >= cols as well as words beyond ceil(cols / 64) are zero.
 *  - Arguments are validated on the host before anything is enqueued; an
 *    invalid call returns an error status and enqueues nothing.  Device-side
 *    faults (e.g. a column index out of range) are not detected; they surface
 *    at the caller's next synchronisation.  Inputs must be finite.
 *  - Calls share no mutable global state: concurrent calls on different
 *    streams with disjoint outputs and workspaces are safe.
 */
#ifndef BIGCN_H
#define BIGCN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BIGCN_OK = 0,
  BIGCN_EINVAL = -1,       /* bad pointer, size or enum value              */
  BIGCN_EALIGN = -2,       /* pointer or leading dimension misaligned      */
  BIGCN_EWORKSPACE = -3,   /* workspace missing or too small               */
  BIGCN_EUNSUPPORTED = -4, /* valid request the library does not implement */
  BIGCN_EHIP = -5          /* the HIP runtime refused a launch             */
} bigcn_status;

/* Storage of the binary-GEMM integer result.  All three hold every value
 * exactly: I32 always, I16 for K <= 32767, F16 (IEEE half) for K <= 2048. */
typedef enum { BIGCN_I32 = 0, BIGCN_I16 = 1, BIGCN_F16 = 2 } bigcn_itype;

/* Normalised adjacency built from the CSR of Â = A + I (Sec. 3.1):
 *   SYM:  Ã = D̂^-1/2 Â D̂^-1/2   (Eq. (1))
 *   MEAN: Ã = D̂^-1 Â            (mean over the closed neighbourhood)
 * where D̂_ii is the number of entries of row i. */
typedef enum { BIGCN_NORM_SYM = 0, BIGCN_NORM_MEAN = 1 } bigcn_norm;

/* Output activation.  Bi-GCN uses none (the next layer's binarisation acts
 * as the non-linearity, Sec. 4.1); ReLU is offered for other uses. */
typedef enum { BIGCN_ACT_NONE = 0, BIGCN_ACT_RELU = 1 } bigcn_act;

/* Binary-GEMM algorithm.  POPCOUNT: XOR + bit count on the vector ALUs.
 * MFMA_I8: the signs expanded to {0,1} bytes and multiplied on the matrix
 * cores (int8 in, int32 accumulate), the +-1 product recovered exactly as
 * 4*sum(ab) - 2*sum(a) - 2*sum(b) + K; N <= 256.  Both give identical
 * results.  AUTO takes MFMA_I8 for M >= 65536 rows with K >= 256 (where it
 * measured faster on MI355X) and POPCOUNT otherwise. */
typedef enum {
  BIGCN_BGEMM_AUTO = 0,
  BIGCN_BGEMM_POPCOUNT = 1,
  BIGCN_BGEMM_MFMA_I8 = 2
} bigcn_bgemm_algo;

/* ---------------------------------------------------------------------------
 * bigcn_binarize_pack -- sign binarisation with per-row scale.
 * Eqs. (7)-(8) for node features (one bucket per row of H); Eqs. (3)-(4)
 * for weights when called on W^T (row j of W^T = column j of W).
 *
 *   x      [rows][ldx] fp32; the first `cols` elements of each row are used.
 *   mu, rstd  both NULL, or both fp32[cols]: the row is first standardised,
 *          y = (x - mu[c]) * rstd[c], as two separately rounded fp32
 *          operations (the input batch normalisation of the paper's set-up,
 *          Sec. 6.2, at inference).  Otherwise y = x.
 *   rowptr NULL, or int64[rows + 1] row pointers of the CSR of Â (one row per
 *          node).  With norm == BIGCN_NORM_SYM the scale is multiplied by
 *          D̂_rr^-1/2 (the source-side factor of Ã); with MEAN it is not.
 *   bits   [rows][ldw] uint64 output, ldw >= ceil(cols / 64); pad bits and
 *          pad words are written as zero.  16-byte aligned if ldw is even.
 *   scale  fp32[rows] output: mean_c |y[r][c]| (times D̂_rr^-1/2, see above).
 *          This is β of Eq. (7) (α of Eq. (4) for weights) with the bucket
 *          length cols as divisor.
 * Errors: EINVAL (NULL x/bits/scale, rows < 0, cols < 1, ldx < cols,
 *         ldw < ceil(cols/64), only one of mu/rstd, bad norm),
 *         EALIGN (x not 4-byte aligned, bits not 8-byte aligned).
 * ------------------------------------------------------------------------- */
bigcn_status bigcn_binarize_pack(const float* x, int64_t rows, int32_t cols,
                                 int64_t ldx, const float* mu,
                                 const float* rstd, const int64_t* rowptr,
                                 bigcn_norm norm, uint64_t* bits, int64_t ldw,
                                 float* scale, void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_bgemm -- binary GEMM of packed sign rows, the ±1 inner products of
 * Eqs. (11)-(12) computed with XOR and bit count:
 *     C[i][j] = K - 2 * popcount(F_i XOR B_j) = sum_k s(F_i,k) * s(B_j,k)
 *
 *   F   [M][ldf] uint64 packed rows (node features), ldf >= ceil(K/64).
 *   B   [N][ldb] uint64 packed rows (weights: rows of W^T), ldb >= ceil(K/64).
 *   K   number of valid sign positions (d_in); pad bits must be zero.
 *   C   [M][ldc] output of type ctype, ldc >= N.
 *   algo  see bigcn_bgemm_algo.
 * Errors: EINVAL (NULL pointers, M < 0, N < 1, K < 1, short leading
 *         dimensions, ctype that cannot hold K: I16 needs K <= 32767, F16
 *         needs K <= 2048), EALIGN (F, B not 8-byte aligned; C not aligned to
 *         its element size), EUNSUPPORTED (K > 8192, or MFMA_I8 for a shape
 *         that variant does not cover).
 * ------------------------------------------------------------------------- */
bigcn_status bigcn_bgemm(const uint64_t* F, int64_t M, int64_t ldf,
                         const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                         void* C, bigcn_itype ctype, int64_t ldc,
                         bigcn_bgemm_algo algo, void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_spmm_csr -- aggregation of Eq. (13) with the rescale of Eq. (11):
 *     out[i][k] = act( rowfac_i * alpha[k] * sum_{e in row i} g[col_e] * C[col_e][k]
 *                      + bias[k] )
 * with rowfac_i = D̂_ii^-1/2 (SYM) or D̂_ii^-1 (MEAN), D̂_ii = rowptr[i+1] -
 * rowptr[i].  With g = β·D̂^-1/2 (SYM) or g = β (MEAN), as written by
 * bigcn_binarize_pack with rowptr, this is out = act(Ã ζ + b),
 * ζ_jk = β_j α_k C_jk.  A row with no entries gives act(bias[k]).
 *
 *   rowptr  int64[n + 1], non-decreasing, rowptr[0] = 0 (CSR of Â).
 *   colidx  int32[rowptr[n]], each in [0, n).
 *   g       fp32[n] per-source-node scale.
 *   C       [n][ldc] integer products of type ctype, ldc >= d, ldc a
 *           multiple of 4, C aligned to 4 elements.
 *   alpha   fp32[d]; bias fp32[d] or NULL.
 *   out     [n][ldo] fp32, ldo >= d.
 *   workspace  device memory of at least bigcn_spmm_workspace_bytes(n,
 *           rowptr_last, d) bytes, 256-byte aligned; contents on entry are
 *           ignored.  nnz (= rowptr[n]) must be passed on the host.
 * Sums run in fp32 in a fixed order: results are bitwise reproducible.
 * Errors: EINVAL, EALIGN (C not aligned to 4 elements, out / g / alpha /
 *         bias not 4-byte aligned, workspace not 256-byte aligned),
 *         EWORKSPACE.
 * ------------------------------------------------------------------------- */
size_t bigcn_spmm_workspace_bytes(int64_t n, int64_t nnz, int32_t d);
bigcn_status bigcn_spmm_csr(int64_t n, int64_t nnz, const int64_t* rowptr,
                            const int32_t* colidx, bigcn_norm norm,
                            const float* g, const void* C, bigcn_itype ctype,
                            int32_t d, int64_t ldc, const float* alpha,
                            const float* bias, bigcn_act act, float* out,
                            int64_t ldo, void* workspace, size_t ws_bytes,
                            void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_bgemm_q8 / bigcn_spmm_csr_q8 -- the binary GEMM and the aggregation
 * with the products kept as exact 8-bit half-codes (half the bytes the
 * aggregation gathers per edge).  Since dot = K - 2 popcount(...) has the
 * parity p = K mod 2, the code (dot - p) / 2 represents every |dot| <= 255
 * in one signed byte.  A row i with a larger |dot| in any column is written
 * in full, exactly (IEEE half), to C16 and flagged by setting the sign bit of
 * g[i]; the aggregation then reads that row from C16.  g is therefore
 * in/out for bigcn_bgemm_q8: it must hold the non-negative scales written by
 * bigcn_binarize_pack, and is left with the flags for bigcn_spmm_csr_q8.
 * Inputs and outputs otherwise as bigcn_bgemm / bigcn_spmm_csr.
 *
 * Row width: NB = 1, 2 or 4 bytes per lane for N (d for the aggregation)
 * of at most 64, 128 or 256 columns; a row spans W = 64 * NB entries.
 *   C8   [M][ldc8] int8, ldc8 >= W and a multiple of 4.  Row order is
 *        lane-interleaved: column k sits at position NB*(k % 64) + k / 64
 *        (the 64 lanes of a wave each find their columns l, l+64, ... in
 *        one NB-byte word); for N <= 64 that is the natural order.
 *   C16  [M][ldc16] IEEE half, ldc16 >= W and a multiple of 4, the same
 *        interleaved order; only flagged rows are written.
 *   g    fp32[M] (see above).
 * Shapes: 1 <= N <= 256, K <= 2048, M * W and M * W * 2 below 4 GiB; other
 * shapes return EUNSUPPORTED (use the exact-type calls).
 * The aggregation result equals bigcn_spmm_csr on the exact products up to
 * fp32 rounding (the sum is formed as 2 * sum g code + p * sum g).
 * ------------------------------------------------------------------------- */
bigcn_status bigcn_bgemm_q8(const uint64_t* F, int64_t M, int64_t ldf,
                            const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                            int8_t* C8, int64_t ldc8, void* C16, int64_t ldc16,
                            float* g, void* stream);
bigcn_status bigcn_spmm_csr_q8(int64_t n, int64_t nnz, const int64_t* rowptr,
                               const int32_t* colidx, bigcn_norm norm,
                               const float* g, const int8_t* C8, int64_t ldc8,
                               const void* C16, int64_t ldc16, int32_t K,
                               int32_t d, const float* alpha, const float* bias,
                               bigcn_act act, float* out, int64_t ldo,
                               void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_spmm_csr_q8_noalloc -- bigcn_spmm_csr_q8 without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that must not call hipMalloc, harnesses that forbid
 * it).  It allocates nothing and calls no allocating routine: its scratch
 * (per-chunk partial rows) lives in a static device array of
 * bigcn_spmm_csr_q8_noalloc_max_bytes() bytes (64.25 MiB) that every GPU the
 * library runs on holds until the process ends.  The first call on a device
 * looks up that device's copy (hipGetSymbolAddress).
 *
 * Arguments, layouts and results as bigcn_spmm_csr_q8.  Graphs of up to
 * 67,108,864 CSR entries are cut into the same chunks as there, so the
 * results are identical; larger graphs are cut into at most 32768 longer
 * chunks (the same sums in another grouping, equal up to fp32 rounding).
 * Calls on one GPU share its scratch array: calls that overlap in time on
 * one GPU (different streams, or host threads) race and must not be issued;
 * calls ordered on one stream are safe.  The array keeps the last call's
 * contents; nothing in it is read before it is written within a call.
 * Errors: as bigcn_spmm_csr_q8, plus EWORKSPACE if the scratch this call
 *         needs exceeds the array (it does not for d <= 256) and EHIP if the
 *         array's device address cannot be obtained.
 * ------------------------------------------------------------------------- */
size_t bigcn_spmm_csr_q8_noalloc_max_bytes(void);
bigcn_status bigcn_spmm_csr_q8_noalloc(int64_t n, int64_t nnz, const int64_t* rowptr,
                                       const int32_t* colidx, bigcn_norm norm,
                                       const float* g, const int8_t* C8, int64_t ldc8,
                                       const void* C16, int64_t ldc16, int32_t K,
                                       int32_t d, const float* alpha, const float* bias,
                                       bigcn_act act, float* out, int64_t ldo,
                                       void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_spmm_csr_sage_q8 -- aggregation of a binarised two-weight GraphSAGE
 * layer with the mean aggregator.  The paper binarises every feature-
 * extraction step of the GNNs it generalises (Sec. 6, Table 3, whose model
 * sizes count a self and a neighbour matrix); both products are formed
 * before aggregating, as in Eq. (13):
 *   out[i][k] = act( alpha_neigh[k] / |N(i)| * sum_{j in N(i)} g[j] dot_n[j][k]
 *                    + |g[i]| * alpha_self[k] * dot_s[i][k] + b_k )
 * with N(i) row i of the CSR given (the graph A, normally without
 * self-loops; an empty row has no neighbour term), g the scales of
 * bigcn_binarize_pack with norm MEAN (beta), flagged by bigcn_bgemm_q8 for
 * the neighbour products C8 / C16 exactly as for bigcn_spmm_csr_q8, and
 * dot_s the node's own products with the self weights:
 *   Cself  [n][ldself] IEEE half, ldself >= d, natural column order (as
 *          written by bigcn_bgemm with ctype F16), 2-byte aligned.
 *   alpha_self  fp32[d].
 * Errors: as bigcn_spmm_csr_q8, plus EINVAL for a NULL Cself / alpha_self
 *         or ldself < d.
 * ------------------------------------------------------------------------- */
bigcn_status bigcn_spmm_csr_sage_q8(int64_t n, int64_t nnz, const int64_t* rowptr,
                                    const int32_t* colidx, const float* g,
                                    const int8_t* C8, int64_t ldc8, const void* C16,
                                    int64_t ldc16, int32_t K, int32_t d,
                                    const float* alpha_neigh, const void* Cself,
                                    int64_t ldself, const float* alpha_self,
                                    const float* bias, bigcn_act act, float* out,
                                    int64_t ldo, void* workspace, size_t ws_bytes,
                                    void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_layer_backward -- back propagation of one binarised graph-convolution
 * layer (Alg. 1 with Eqs. (14)-(15); training is outside the forward path,
 * this is the gradient the paper's algorithm defines):
 *   G     = gout, masked by 1[out > 0] when act is RELU
 *   db    = sum_i G_i                       dζ = Ã^T G
 *   dW~   = H~^T dζ,   H~ = diag(β) sign(H) (Eqs. (7)-(8))
 *   dH~   = dζ W~^T,   W~ = sign(W) diag(α) (Eqs. (3)-(4))
 *   dH    = dH~ * 1[|dH~| < 1]              (Eq. (14), the indicator taken
 *                                            on |dH~| as printed)
 *   dW_ij = B_ij / d_in * sum_k dW~_kj B_kj + α_j dW~_ij 1[|W_ij| < 1]
 *                                           (Eq. (15), straight-through
 *                                            estimator for sign)
 * The CSR of Â must be structurally symmetric (an undirected graph with its
 * self-loops, as for the forward); Ã and its normalisation as for
 * bigcn_spmm_csr.
 *   slot, colslot  the source order of bigcn_source_slots, or both NULL.
 *          When given, G and the source factors are staged in that order
 *          and dζ gathers them through colslot (the same terms in the same
 *          order: every result is identical either way).
 *   h      [n][ldh] fp32 layer input (before binarisation), ldh >= d_in
 *   wt     [d_out][ldwt] fp32 W^T; wbits [d_out][ldw], alpha fp32[d_out]:
 *          W^T packed by bigcn_binarize_pack
 *   gout   [n][ldg] fp32 dL/dH^(l+1); out [n][ldo] the forward output of
 *          the layer (read for RELU only, may be NULL otherwise)
 *   dwt    [d_out][lddw] fp32 dL/dW in the W^T layout (required)
 *   dh, dh_tilde  [n][ld] fp32 dL/dH and dL/dH~, each nullable
 *   dwt_tilde [d_out][lddwt] fp32 dL/dW~ (W^T layout), db fp32[d_out],
 *          dzeta [n][lddz] fp32 dL/dζ: each nullable
 *   workspace  bigcn_layer_backward_workspace_bytes(n, nnz, d_in, d_out)
 *          bytes, 256-byte aligned; contents on entry are ignored.
 * Sums over nodes (db, dW~) are formed in fp64 over fixed chunks of rows
 * and added in order; every result is reproducible bit for bit.
 * Errors: EINVAL (bad sizes, NULL required pointers, short leading
 *         dimensions, bad norm / act, only one of slot / colslot), EALIGN
 *         (pointers not aligned to their element size, workspace not
 *         256-byte aligned), EWORKSPACE, EUNSUPPORTED (d_in > 2048 or
 *         d_out > 256).
 * ------------------------------------------------------------------------- */
size_t bigcn_layer_backward_workspace_bytes(int64_t n, int64_t nnz, int32_t d_in,
                                            int32_t d_out);
bigcn_status bigcn_layer_backward(int64_t n, int64_t nnz, const int64_t* rowptr,
                                  const int32_t* colidx, const int32_t* slot,
                                  const int32_t* colslot, bigcn_norm norm, const float* h,
                                  int64_t ldh, int32_t d_in, const float* wt, int64_t ldwt,
                                  const uint64_t* wbits, int64_t ldw, const float* alpha,
                                  int32_t d_out, const float* gout, int64_t ldg,
                                  const float* out, int64_t ldo, bigcn_act act,
                                  float* dh, int64_t lddh, float* dh_tilde,
                                  int64_t lddht, float* dwt, int64_t lddw,
                                  float* dwt_tilde, int64_t lddwt, float* db,
                                  float* dzeta, int64_t lddz, void* workspace,
                                  size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_source_slots -- the source order bigcn_forward can store its
 * per-node products and scales in (built once per graph, like the CSR).
 * The aggregation of Eq. (13) reads one source row per edge; in a power-law
 * graph most edges lead to a few high-degree nodes.  Listing nodes by
 * descending degree class (class 0 for degree <= 1, else floor(log2
 * degree)), by node id within a class, puts those nodes' rows and scales
 * together in memory, so more of the gathers hit cache.
 *   rowptr, colidx  the graph (as for bigcn_spmm_csr; degree = row count).
 *   slot     int32[n] output: node i's position in that order.
 *   colslot  int32[nnz] output: slot[colidx[e]].
 *   workspace  bigcn_source_slots_workspace_bytes(n) bytes, 256-byte
 *            aligned; contents on entry are ignored.
 * Errors: EINVAL (n < 0, nnz < 0, n > INT32_MAX, NULL rowptr / slot with
 *         n > 0, NULL colidx / colslot with nnz > 0), EALIGN, EWORKSPACE.
 * ------------------------------------------------------------------------- */
size_t bigcn_source_slots_workspace_bytes(int64_t n);
bigcn_status bigcn_source_slots(int64_t n, int64_t nnz, const int64_t* rowptr,
                                const int32_t* colidx, int32_t* slot, int32_t* colslot,
                                void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_forward -- the whole multi-layer forward pass (Sec. 4.1):
 *     H^(0) = X,  H^(l+1) = act_l( Ã ζ^(l) + b_l ),  l = 0 .. n_layers-1,
 * every layer binarised (features and weights).  Layer 0 standardises X with
 * mu / rstd when given (see bigcn_binarize_pack).
 *
 * One layer description per layer (HOST array of n_layers entries; the
 * pointers inside are device pointers):
 *   d_in, d_out  layer widths; layers[l+1].d_in must equal layers[l].d_out.
 *   wbits  [d_out][ldw] packed signs of W^T, ldw >= ceil(d_in/64)
 *   alpha  fp32[d_out]   (both as written by bigcn_binarize_pack on W^T)
 *   bias   fp32[d_out] or NULL;  act  output activation of the layer.
 *
 *   n, nnz, rowptr, colidx, norm   the graph, as for bigcn_spmm_csr.
 *   slot, colslot  both NULL, or the source order of bigcn_source_slots
 *        (device int32[n] and int32[nnz]): slot a permutation of [0, n),
 *        colslot[e] = slot[colidx[e]].  Each layer then stores node i's
 *        products and scale at row slot[i] of its internal buffers and the
 *        aggregations gather by colslot; inputs and outputs keep the node
 *        order, every sum keeps its terms and their order, and the result
 *        is bit-identical to the call without them.  Ignored when nnz = 0.
 *   x    [n][ldx] fp32 node features, ldx >= layers[0].d_in.
 *   out  [n][ldo] fp32 result of the last layer, ldo >= last d_out.
 *   workspace  at least bigcn_forward_workspace_bytes(...) bytes for the
 *          same layers (a hidden output the caller gives needs no workspace
 *          copy), 256-byte aligned; contents on entry are ignored.
 * Internally each layer's products are kept exactly: as 8-bit half-codes
 * (see bigcn_bgemm_q8) for layers of up to 256 output columns with
 * d_in <= 2048, otherwise in IEEE half (d_in <= 2048) or int16.  When two
 * consecutive layers both use 8-bit codes, the second layer's sign pack and
 * binary GEMM run inside the aggregation that produces its input: the
 * hidden activations are not written to memory unless the layer gives an
 * output (bigcn_layer.out).  The result is
 * bit-identical to chaining the per-step entry points (bigcn_binarize_pack,
 * bigcn_bgemm_q8, bigcn_spmm_csr_q8 for 8-bit layers).
 * A layer with wbits_self set is a two-weight GraphSAGE layer: the graph
 * given is then A (the neighbour sets, normally without self-loops) and
 * norm must be MEAN; its products stay unfused (8-bit neighbour codes, then
 * bigcn_spmm_csr_sage_q8's aggregation; the self products are formed in the
 * aggregation's epilogue from the packed signs for 65-256 output columns,
 * else read as exact half products).
 * Errors: as the per-step calls, plus EINVAL for inconsistent layer widths
 *         or n_layers < 1, only one of slot / colslot, or a GraphSAGE layer
 *         with norm SYM, EALIGN for slot / colslot not 4-byte aligned,
 *         EUNSUPPORTED
 *         for d_in > 8192 on a layer or a GraphSAGE layer outside the 8-bit
 *         shapes (d_out <= 256, d_in <= 2048).
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t d_in;
  int32_t d_out;
  const uint64_t* wbits;
  int64_t ldw;
  const float* alpha;
  const float* bias;
  bigcn_act act;
  /* NULL for a graph-convolution layer.  Otherwise the layer is a two-weight
   * GraphSAGE layer (see bigcn_spmm_csr_sage_q8): wbits / alpha are the
   * neighbour weights, these the self weights, packed the same way. */
  const uint64_t* wbits_self;
  int64_t ldw_self;
  const float* alpha_self;
  /* NULL, or where this hidden layer's fp32 output H^(l+1) [n][ldo] is
   * written as well (ldo >= d_out, 4-byte aligned, overlapping no other
   * argument); ignored for the last layer, whose output is bigcn_forward's
   * out.  Without it a layer whose aggregation forms the next layer's
   * products in its epilogue writes no fp32 output at all. */
  float* out;
  int64_t ldo;
} bigcn_layer;

size_t bigcn_forward_workspace_bytes(int64_t n, int64_t nnz,
                                     const bigcn_layer* layers,
                                     int32_t n_layers);
bigcn_status bigcn_forward(int64_t n, int64_t nnz, const int64_t* rowptr,
                           const int32_t* colidx, const int32_t* slot,
                           const int32_t* colslot, bigcn_norm norm,
                           const float* x, int64_t ldx, const float* mu,
                           const float* rstd, const bigcn_layer* layers,
                           int32_t n_layers, float* out, int64_t ldo,
                           void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * bigcn_check_csr -- validates the contents of a CSR graph on the device
 * (the entry points above take them on trust: a bad row pointer or column
 * index there is an out-of-range access).  The graph is the input every
 * aggregation reads (Sec. 3.1: the rows of Â, or of A for the GraphSAGE
 * layer); a caller checks it once, before its first use.
 *
 *   n, nnz   rows and entries (host values).
 *   rowptr   int64[n + 1] (device), colidx int32[nnz] (device); only read,
 *            each element once, at positions < n + 1 and < nnz.
 *   flags    int32[1] (device, caller-owned): set to the OR of
 *              1  rowptr[0] != 0
 *              2  rowptr[n] != nnz
 *              4  rowptr decreases somewhere
 *              8  a column index outside [0, n)
 *            and 0 for a valid graph.  Ready when `stream` is synchronised.
 * Errors: EINVAL (n < 0, nnz < 0, n > INT32_MAX, NULL flags, NULL rowptr,
 *         or NULL colidx with nnz > 0), EALIGN, EHIP.
 * ------------------------------------------------------------------------- */
bigcn_status bigcn_check_csr(int64_t n, int64_t nnz, const int64_t* rowptr,
                             const int32_t* colidx, int32_t* flags, void* stream);

/* Human-readable text of a status code (static storage, never NULL). */
const char* bigcn_status_string(bigcn_status s);

#ifdef __cplusplus
}
#endif

#endif /* BIGCN_H */
