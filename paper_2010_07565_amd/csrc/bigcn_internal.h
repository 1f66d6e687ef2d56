// Internal launch interface between the C ABI layer (bigcn_api.hip) and the
// gfx950 kernels (bigcn_kernels.hip).  Arguments are validated by the ABI
// layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bigcn {

// Element storage of binary-GEMM products (same values as bigcn_itype), and
// fp32 rows for the aggregation of gradients (internal only).
enum class IType : int { I32 = 0, I16 = 1, F16 = 2, F32 = 3 };

inline size_t itype_size(IType t) { return (t == IType::I32 || t == IType::F32) ? 4 : 2; }

// Sign-pack rows of x; see bigcn_binarize_pack.  sym != 0 folds D̂^-1/2 into
// the scale when rowptr is given.  With slot (a permutation of [0, rows))
// row r's bits and scale are written to row slot[r] (the source order of
// the forward pass); the degree for D̂ is still row r's.
hipError_t launch_pack(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                       const float* mu, const float* rstd,
                       const int64_t* rowptr, int sym, uint64_t* bits,
                       int64_t ldw, float* scale, hipStream_t stream,
                       const int32_t* slot = nullptr);

// C[i][j] = K - 2 popcount(F_i ^ B_j) on the vector ALUs.
hipError_t launch_bgemm_popcount(const uint64_t* F, int64_t M, int64_t ldf,
                                 const uint64_t* B, int32_t N, int64_t ldb,
                                 int32_t K, void* C, IType ct, int64_t ldc,
                                 hipStream_t stream);

// The same product with +-1 int8 operands on the matrix cores.
bool bgemm_mfma_supported(int32_t N, int32_t K);
hipError_t launch_bgemm_mfma(const uint64_t* F, int64_t M, int64_t ldf,
                             const uint64_t* B, int32_t N, int64_t ldb,
                             int32_t K, void* C, IType ct, int64_t ldc,
                             hipStream_t stream);

// Exact 8-bit half-code storage of the products (layers of up to 256 output
// columns with K <= 2048): codes (dot - K%2)/2 in C8 rows of 64*NB bytes,
// NB = q8_lane_bytes(N), in lane-interleaved order (column k at byte
// NB*(k%64) + k/64); rows with |dot| > 255 written exactly (half, same
// order, 64*NB per row) to C16 and flagged by the sign bit of g.
constexpr int q8_lane_bytes(int32_t N) { return N <= 64 ? 1 : N <= 128 ? 2 : 4; }
bool q8_supported(int64_t n, int32_t N, int32_t K);
// The pack of a layer's input followed, in the same kernel, by its binary
// GEMM into 8-bit half-codes (layers of N <= 256 outputs with
// ceil(K / 64) * q8_lane_bytes(N) <= 16: up to 1024 inputs for 64 outputs,
// 512 for 128, 256 for 256; row stride at most 2^24 elements): the codes,
// exact rows and flagged scale of launch_pack + launch_bgemm_q8, bit for
// bit, without writing the packed bits.
bool pack_bgemm_q8_supported(int32_t cols, int32_t N, int64_t ldx);
hipError_t launch_pack_bgemm_q8(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                                const float* mu, const float* rstd, const int64_t* rowptr,
                                int sym, const uint64_t* B, int32_t N, int64_t ldb,
                                int8_t* C8, int64_t ldc8, void* C16, int64_t ldc16,
                                float* g, hipStream_t stream,
                                const int32_t* slot = nullptr);
hipError_t launch_bgemm_q8(const uint64_t* F, int64_t M, int64_t ldf,
                           const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                           int8_t* C8, int64_t ldc8, void* C16, int64_t ldc16,
                           float* g, hipStream_t stream);

// A next layer fused into the 8-bit aggregation's epilogue: the finished
// output rows are binarised and multiplied with the next weights in place.
//   kind 0: none (the output rows are written);
//   kind 1: next products as 8-bit half-codes (C8, C16 fallback, flags in g),
//           rows of 64*q8_lane_bytes(d_out) codes / halves.
//   kind 2: no next layer; the rows get the self term of a two-weight
//           GraphSAGE layer, |g_i| alpha_self[k] Cself[i][k], before bias and
//           activation (Cself: exact half products with the self weights).
//   kind 3: as kind 2, the self products formed in the epilogue from the
//           layer's own packed signs F (row i at F + i ldF, the rows the
//           aggregation's g and products use) and the self weights' packed
//           W^T (wself [d][ldw_self], kin inputs) instead of read from Cself;
//           see self_in_epilogue_supported.
// g receives the next layer's per-node scale.
struct FusedNext {
  int kind;
  const uint64_t* wbits;  // next layer's packed W^T [d_out][ldw]
  int64_t ldw;
  int32_t d_out;
  int8_t* C8;
  int64_t ldc8;
  void* C16;
  int64_t ldc16;
  float* g;
  const void* Cself;      // kind 2
  int64_t ldself;
  const float* alpha_self;
  // Source order (nullable): row r's next-layer products (kind 1) or self
  // products and scale (kinds 2, 3) sit at row slot[r].
  const int32_t* slot;
  const uint64_t* F;      // kind 3
  int64_t ldF;
  const uint64_t* wself;
  int64_t ldw_self;
  int32_t kin;
};
// Layers whose self term kind 3 can form: the wide 8-bit aggregation (65-256
// outputs) with the self weights' words per lane, ceil(kin / 64) times
// q8_lane_bytes(d), at most 16 (kin <= 256 for 129-256 outputs, <= 512 for
// 65-128), staged in LDS.
bool self_in_epilogue_supported(int64_t nnz, int32_t d, int32_t kin);

// Aggregation over the CSR of Â with the fused rescale / bias / activation
// epilogue.  The edge range [0, nnz) is cut into fixed chunks of `chunk`
// edges; see bigcn_kernels.hip for the scheme and the workspace layout.
struct SpmmPlan {
  int64_t chunk;      // edges per worker
  int64_t workers;    // ceil(nnz / chunk), at least 1
  int32_t dpad;       // columns per partial row (multiple of 4)
  size_t bytes;       // workspace bytes
  size_t off_rowof, off_tailrow, off_head, off_tail;
};
// max_workers caps the number of workers (chunks grow past 2048 edges when
// needed), which bounds the workspace for a fixed-size scratch buffer.
SpmmPlan spmm_plan(int64_t n, int64_t nnz, int32_t d, int64_t max_workers = INT64_MAX);

// Builds the per-worker start rows (once per graph and chunk size).
hipError_t launch_spmm_rows(int64_t n, int64_t nnz, const int64_t* rowptr,
                            const SpmmPlan& plan, void* workspace,
                            hipStream_t stream);
// Aggregation proper; requires launch_spmm_rows to have run on `workspace`.
// mean: 0 symmetric, 1 mean, 2 no destination factor (see row_factor_deg).
hipError_t launch_spmm(int64_t n, int64_t nnz, const int64_t* rowptr,
                       const int32_t* colidx, int mean, const float* g,
                       const void* C, IType ct, int32_t d, int64_t ldc,
                       const float* alpha, const float* bias, int relu,
                       float* out, int64_t ldo, const SpmmPlan& plan,
                       void* workspace, hipStream_t stream);

// Aggregation reading 8-bit half-codes (see launch_bgemm_q8; needs no row
// plan: launch_spmm_rows is not required); with a
// FusedNext of kind > 0 the output rows feed the next layer instead of (or,
// if out != nullptr, besides) being written.
hipError_t launch_spmm_q8(int64_t n, int64_t nnz, const int64_t* rowptr,
                          const int32_t* colidx, int mean, const float* g,
                          const int8_t* C8, int64_t ldc8, const void* C16,
                          int64_t ldc16, int32_t K, int32_t d, const float* alpha,
                          const float* bias, int relu, float* out, int64_t ldo,
                          const SpmmPlan& plan, void* workspace,
                          const FusedNext* next, hipStream_t stream);

// Source order of the forward pass (see bigcn_source_slots): slot[i] for
// every node, colslot[e] = slot[colidx[e]]; workspace of SlotPlan::bytes.
struct SlotPlan {
  int64_t groups;   // groups of 64 nodes
  int64_t total;    // class counts, 32 per group
  int64_t blocks;   // scan blocks of 1024 counts
  size_t off_sums;  // byte offset of the block sums
  size_t bytes;
};
SlotPlan source_slots_plan(int64_t n);
hipError_t launch_source_slots(int64_t n, int64_t nnz, const int64_t* rowptr,
                               const int32_t* colidx, int32_t* slot, int32_t* colslot,
                               void* workspace, hipStream_t stream);

}  // namespace bigcn
