// C ABI of the binarized-GCN library: host-side argument validation and the
// multi-layer forward orchestration.  Every entry point validates on the host
// and then only enqueues kernels on the caller's stream.

#include <stdint.h>

#include <algorithm>
#include <mutex>

#include "../../include/bigcn.h"
#include "bigcn_internal.h"

namespace {

using bigcn::IType;

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }
inline int64_t words(int64_t k) { return (k + 63) / 64; }
constexpr size_t up256(size_t v) { return (v + 255) & ~(size_t)255; }

inline bool itype_ok(int t) { return t == BIGCN_I32 || t == BIGCN_I16 || t == BIGCN_F16; }
inline bool itype_holds(int t, int64_t K) {
  return t == BIGCN_I32 || (t == BIGCN_I16 && K <= 32767) || (t == BIGCN_F16 && K <= 2048);
}
// Exact storage used inside the forward pass for a layer of width K.
inline IType forward_itype(int64_t K) {
  return K <= 2048 ? IType::F16 : (K <= 32767 ? IType::I16 : IType::I32);
}

inline bigcn_status hip_status(hipError_t e) { return e == hipSuccess ? BIGCN_OK : BIGCN_EHIP; }

constexpr int32_t kMaxBgemmK = 8192;

bigcn_status check_pack(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                        const float* mu, const float* rstd, int norm,
                        const uint64_t* bits, int64_t ldw, const float* scale) {
  if (rows < 0 || cols < 1 || ldx < cols || ldw < words(cols)) return BIGCN_EINVAL;
  if ((mu == nullptr) != (rstd == nullptr)) return BIGCN_EINVAL;
  if (norm != BIGCN_NORM_SYM && norm != BIGCN_NORM_MEAN) return BIGCN_EINVAL;
  if (rows > 0 && (x == nullptr || bits == nullptr || scale == nullptr)) return BIGCN_EINVAL;
  if (!aligned(x, 4) || !aligned(bits, 8) || !aligned(scale, 4)) return BIGCN_EALIGN;
  if (mu != nullptr && (!aligned(mu, 4) || !aligned(rstd, 4))) return BIGCN_EALIGN;
  return BIGCN_OK;
}

bigcn_status check_bgemm(const uint64_t* F, int64_t M, int64_t ldf,
                         const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                         const void* C, int ctype, int64_t ldc, int algo) {
  if (M < 0 || N < 1 || K < 1) return BIGCN_EINVAL;
  if (ldf < words(K) || ldb < words(K) || ldc < N) return BIGCN_EINVAL;
  if (!itype_ok(ctype) || !itype_holds(ctype, K)) return BIGCN_EINVAL;
  if (algo != BIGCN_BGEMM_AUTO && algo != BIGCN_BGEMM_POPCOUNT && algo != BIGCN_BGEMM_MFMA_I8)
    return BIGCN_EINVAL;
  if (B == nullptr || (M > 0 && (F == nullptr || C == nullptr))) return BIGCN_EINVAL;
  if (!aligned(F, 8) || !aligned(B, 8) || !aligned(C, bigcn::itype_size((IType)ctype)))
    return BIGCN_EALIGN;
  if (K > kMaxBgemmK) return BIGCN_EUNSUPPORTED;
  return BIGCN_OK;
}

bigcn_status check_graph(int64_t n, int64_t nnz, const int64_t* rowptr,
                         const int32_t* colidx, int norm) {
  if (n < 0 || nnz < 0 || n > INT32_MAX) return BIGCN_EINVAL;
  if (norm != BIGCN_NORM_SYM && norm != BIGCN_NORM_MEAN) return BIGCN_EINVAL;
  if (n > 0 && rowptr == nullptr) return BIGCN_EINVAL;
  if (nnz > 0 && colidx == nullptr) return BIGCN_EINVAL;
  if (!aligned(rowptr, 8) || !aligned(colidx, 4)) return BIGCN_EALIGN;
  return BIGCN_OK;
}

bigcn_status check_spmm_operands(int64_t n, const float* g, const void* C,
                                 int ctype, int32_t d, int64_t ldc,
                                 const float* alpha, const float* bias,
                                 int act, const float* out, int64_t ldo) {
  if (d < 1 || ldc < d || ldo < d || (ldc % 4) != 0) return BIGCN_EINVAL;
  if (!itype_ok(ctype)) return BIGCN_EINVAL;
  if (act != BIGCN_ACT_NONE && act != BIGCN_ACT_RELU) return BIGCN_EINVAL;
  if (alpha == nullptr) return BIGCN_EINVAL;
  if (n > 0 && (g == nullptr || C == nullptr || out == nullptr)) return BIGCN_EINVAL;
  if (!aligned(g, 4) || !aligned(C, 4 * bigcn::itype_size((IType)ctype)) ||
      !aligned(out, 4) || !aligned(alpha, 4) || !aligned(bias, 4))
    return BIGCN_EALIGN;
  return BIGCN_OK;
}

// AUTO takes the matrix cores where they measured faster on MI355X: at
// least 64K rows and K >= 256 (a contraction long enough to pay for the
// sign expansion).  With K <= 128 the product write dominates and the
// popcount kernel's wider stores win; below 64K rows both are launch bound.
bool auto_picks_mfma(int64_t M, int32_t N, int32_t K) {
  return bigcn::bgemm_mfma_supported(N, K) && M >= 65536 && K >= 256;
}

hipError_t run_bgemm(const uint64_t* F, int64_t M, int64_t ldf, const uint64_t* B,
                     int32_t N, int64_t ldb, int32_t K, void* C, IType ct,
                     int64_t ldc, int algo, hipStream_t s) {
  const bool mfma = algo == BIGCN_BGEMM_MFMA_I8 ||
                    (algo == BIGCN_BGEMM_AUTO && auto_picks_mfma(M, N, K));
  if (mfma && bigcn::bgemm_mfma_supported(N, K))
    return bigcn::launch_bgemm_mfma(F, M, ldf, B, N, ldb, K, C, ct, ldc, s);
  return bigcn::launch_bgemm_popcount(F, M, ldf, B, N, ldb, K, C, ct, ldc, s);
}

// Workspace layout of bigcn_forward.  Two sets of (scale g, 8-bit codes C8,
// 16-bit products C16) alternate between layers, so a layer can write the
// next layer's products while its own are being read.  ldc8 / ldc16 are the
// capacities per node; an 8-bit layer uses rows of q8_row(d_out).
struct ForwardLayout {
  int64_t ldF, ldh, ldc8, ldc16, ldS;
  size_t off_F, off_g[2], off_C8[2], off_C16[2], off_H0, off_H1, off_S, off_spmm, bytes;
  int32_t dmax;
};

// Whether layer l's aggregation produces layer l+1's products in its
// epilogue (see bigcn::FusedNext): both layers on the 8-bit path.
int fuse_kind(int64_t n, int64_t nnz, const bigcn_layer* layers, int32_t nl, int32_t l) {
  if (l + 1 >= nl || nnz == 0) return 0;
  const bigcn_layer& a = layers[l];
  const bigcn_layer& b = layers[l + 1];
  if (a.wbits_self != nullptr || b.wbits_self != nullptr) return 0;  // GraphSAGE layers
  if (!bigcn::q8_supported(n, a.d_out, a.d_in)) return 0;  // producer: 8-bit wave kernel
  return bigcn::q8_supported(n, b.d_out, b.d_in) ? 1 : 0;
}

// Row stride (bytes of codes, or halves of exact products) of the 8-bit
// layout for a layer of d outputs.
inline int64_t q8_row(int32_t d) { return 64 * bigcn::q8_lane_bytes(d); }

bool forward_layout(int64_t n, int64_t nnz, const bigcn_layer* layers, int32_t nl,
                    ForwardLayout* L) {
  int64_t kwmax = 1, dmax = 1, hmax = 1, smax = 0;
  bool need_h[2] = {false, false};  // a hidden output in workspace set l & 1
  for (int32_t l = 0; l < nl; ++l) {
    kwmax = std::max<int64_t>(kwmax, words(layers[l].d_in));
    dmax = std::max<int64_t>(dmax, layers[l].d_out);
    // a hidden layer writes its fp32 output to the workspace unless its
    // aggregation forms the next layer's products or the caller gives one
    if (l + 1 < nl && layers[l].out == nullptr && fuse_kind(n, nnz, layers, nl, l) == 0) {
      hmax = std::max<int64_t>(hmax, layers[l].d_out);
      need_h[l & 1] = true;
    }
    if (layers[l].wbits_self != nullptr) smax = std::max<int64_t>(smax, layers[l].d_out);
  }
  L->ldS = (smax + 7) / 8 * 8;
  L->ldF = (kwmax + 1) / 2 * 2;
  L->ldh = (hmax + 3) / 4 * 4;
  L->ldc8 = 256;
  L->ldc16 = std::max<int64_t>(256, (dmax + 7) / 8 * 8);
  L->dmax = (int32_t)dmax;
  size_t off = 0;
  L->off_F = off;
  off += up256((size_t)n * L->ldF * 8);
  for (int s = 0; s < 2; ++s) {
    L->off_g[s] = off;
    off += up256((size_t)n * 4);
    L->off_C8[s] = off;
    off += up256((size_t)n * L->ldc8);
    L->off_C16[s] = off;
    off += up256((size_t)n * L->ldc16 * 2);
  }
  L->off_H0 = off;
  if (need_h[0]) off += up256((size_t)n * L->ldh * 4);
  L->off_H1 = off;
  if (need_h[1]) off += up256((size_t)n * L->ldh * 4);
  L->off_S = off;
  off += up256((size_t)n * L->ldS * 2);
  L->off_spmm = off;
  off += bigcn::spmm_plan(n, nnz, (int32_t)dmax).bytes;
  L->bytes = off;
  return true;
}

// Scratch of bigcn_spmm_csr_q8_noalloc: a file-scope device array, one copy
// per GPU, alive until the process ends.  Its size is the largest workspace
// of the 8-bit aggregation with at most kNoallocWorkers workers and rows of
// up to 256 columns (two int32 arrays and two fp32 partial-row arrays of
// kNoallocWorkers entries).  Host code never uses the array's name as an
// address: each device's address comes from hipGetSymbolAddress, taken once
// per device the first time the entry point runs there.
constexpr int64_t kNoallocWorkers = 32768;
constexpr size_t kNoallocScratchBytes =
    2 * up256((size_t)kNoallocWorkers * 4) + 2 * up256((size_t)kNoallocWorkers * 256 * 4);
static __device__ __align__(256) __attribute__((used)) unsigned char
    scratch[kNoallocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (nullptr on failure).
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

namespace {

// Contents of a CSR graph, flags as bigcn_check_csr documents: one kernel
// clears the flags word, the next (stream-ordered after it) ORs in what
// each thread finds; every element is read once, in range.
__global__ void k_csr_clear(int32_t* flags) { *flags = 0; }

__global__ void k_csr_check(int64_t n, int64_t nnz, const int64_t* __restrict__ rowptr,
                            const int32_t* __restrict__ colidx, int32_t* flags) {
  int32_t f = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i <= n || i < nnz;
       i += stride) {
    if (i <= n) {
      const int64_t r = rowptr[i];
      if (i == 0 && r != 0) f |= 1;
      if (i == n && r != nnz) f |= 2;
      if (i < n && rowptr[i + 1] < r) f |= 4;
    }
    if (i < nnz) {
      const int32_t c = colidx[i];
      if (c < 0 || (int64_t)c >= n) f |= 8;
    }
  }
  if (f != 0) atomicOr(flags, f);
}

}  // namespace

extern "C" {

bigcn_status bigcn_check_csr(int64_t n, int64_t nnz, const int64_t* rowptr,
                             const int32_t* colidx, int32_t* flags, void* stream) {
  if (n < 0 || nnz < 0 || n > INT32_MAX || flags == nullptr || rowptr == nullptr ||
      (nnz > 0 && colidx == nullptr))
    return BIGCN_EINVAL;
  if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(flags, 4)) return BIGCN_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(k_csr_clear, dim3(1), dim3(1), 0, s, flags);
  const int64_t items = std::max<int64_t>(n + 1, nnz);
  const int64_t blocks = std::min<int64_t>((items + 255) / 256, 4096);
  hipLaunchKernelGGL(k_csr_check, dim3((unsigned)blocks), dim3(256), 0, s, n, nnz, rowptr,
                     colidx, flags);
  return hipGetLastError() == hipSuccess ? BIGCN_OK : BIGCN_EHIP;
}

const char* bigcn_status_string(bigcn_status s) {
  switch (s) {
    case BIGCN_OK: return "ok";
    case BIGCN_EINVAL: return "invalid argument";
    case BIGCN_EALIGN: return "misaligned pointer or leading dimension";
    case BIGCN_EWORKSPACE: return "workspace missing or too small";
    case BIGCN_EUNSUPPORTED: return "valid request the library does not implement";
    case BIGCN_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

bigcn_status bigcn_binarize_pack(const float* x, int64_t rows, int32_t cols,
                                 int64_t ldx, const float* mu, const float* rstd,
                                 const int64_t* rowptr, bigcn_norm norm,
                                 uint64_t* bits, int64_t ldw, float* scale,
                                 void* stream) {
  bigcn_status st = check_pack(x, rows, cols, ldx, mu, rstd, norm, bits, ldw, scale);
  if (st != BIGCN_OK) return st;
  if (!aligned(rowptr, 8)) return BIGCN_EALIGN;
  return hip_status(bigcn::launch_pack(x, rows, cols, ldx, mu, rstd, rowptr,
                                       norm == BIGCN_NORM_SYM, bits, ldw, scale,
                                       (hipStream_t)stream));
}

bigcn_status bigcn_bgemm(const uint64_t* F, int64_t M, int64_t ldf,
                         const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                         void* C, bigcn_itype ctype, int64_t ldc,
                         bigcn_bgemm_algo algo, void* stream) {
  bigcn_status st = check_bgemm(F, M, ldf, B, N, ldb, K, C, ctype, ldc, algo);
  if (st != BIGCN_OK) return st;
  if (algo == BIGCN_BGEMM_MFMA_I8 && !bigcn::bgemm_mfma_supported(N, K))
    return BIGCN_EUNSUPPORTED;
  return hip_status(run_bgemm(F, M, ldf, B, N, ldb, K, C, (IType)ctype, ldc, algo,
                              (hipStream_t)stream));
}

size_t bigcn_spmm_workspace_bytes(int64_t n, int64_t nnz, int32_t d) {
  if (n < 0 || nnz < 0 || d < 1) return 0;
  return bigcn::spmm_plan(n, nnz, d).bytes;
}

bigcn_status bigcn_spmm_csr(int64_t n, int64_t nnz, const int64_t* rowptr,
                            const int32_t* colidx, bigcn_norm norm,
                            const float* g, const void* C, bigcn_itype ctype,
                            int32_t d, int64_t ldc, const float* alpha,
                            const float* bias, bigcn_act act, float* out,
                            int64_t ldo, void* workspace, size_t ws_bytes,
                            void* stream) {
  bigcn_status st = check_graph(n, nnz, rowptr, colidx, norm);
  if (st != BIGCN_OK) return st;
  st = check_spmm_operands(n, g, C, ctype, d, ldc, alpha, bias, act, out, ldo);
  if (st != BIGCN_OK) return st;
  const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, d);
  if (n > 0 && nnz > 0) {
    if (workspace == nullptr || ws_bytes < plan.bytes) return BIGCN_EWORKSPACE;
    if (!aligned(workspace, 256)) return BIGCN_EALIGN;
  }
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = bigcn::launch_spmm_rows(n, nnz, rowptr, plan, workspace, s);
  if (e != hipSuccess) return BIGCN_EHIP;
  return hip_status(bigcn::launch_spmm(n, nnz, rowptr, colidx,
                                       norm == BIGCN_NORM_MEAN, g, C, (IType)ctype,
                                       d, ldc, alpha, bias, act == BIGCN_ACT_RELU,
                                       out, ldo, plan, workspace, s));
}

bigcn_status bigcn_bgemm_q8(const uint64_t* F, int64_t M, int64_t ldf,
                            const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                            int8_t* C8, int64_t ldc8, void* C16, int64_t ldc16,
                            float* g, void* stream) {
  if (M < 0 || N < 1 || K < 1 || ldf < words(K) || ldb < words(K)) return BIGCN_EINVAL;
  if (ldc8 < q8_row(N) || ldc8 % 4 != 0 || ldc16 < q8_row(N) || ldc16 % 4 != 0)
    return BIGCN_EINVAL;
  if (B == nullptr || (M > 0 && (F == nullptr || C8 == nullptr || C16 == nullptr ||
                                 g == nullptr)))
    return BIGCN_EINVAL;
  if (!aligned(F, 8) || !aligned(B, 8) || !aligned(C8, 4) || !aligned(C16, 8) ||
      !aligned(g, 4))
    return BIGCN_EALIGN;
  if (!bigcn::q8_supported(M, N, K) || (uint64_t)M * ldc8 > 0xFFFFFFFFull ||
      (uint64_t)M * ldc16 * 2 > 0xFFFFFFFFull)
    return BIGCN_EUNSUPPORTED;
  return hip_status(bigcn::launch_bgemm_q8(F, M, ldf, B, N, ldb, K, C8, ldc8, C16, ldc16,
                                           g, (hipStream_t)stream));
}

bigcn_status bigcn_spmm_csr_q8(int64_t n, int64_t nnz, const int64_t* rowptr,
                               const int32_t* colidx, bigcn_norm norm,
                               const float* g, const int8_t* C8, int64_t ldc8,
                               const void* C16, int64_t ldc16, int32_t K,
                               int32_t d, const float* alpha, const float* bias,
                               bigcn_act act, float* out, int64_t ldo,
                               void* workspace, size_t ws_bytes, void* stream) {
  bigcn_status st = check_graph(n, nnz, rowptr, colidx, norm);
  if (st != BIGCN_OK) return st;
  if (K < 1 || d < 1 || ldc8 < q8_row(d) || ldc8 % 4 != 0 || ldc16 < q8_row(d))
    return BIGCN_EINVAL;
  st = check_spmm_operands(n, g, C16, BIGCN_F16, d, ldc16, alpha, bias, act, out, ldo);
  if (st != BIGCN_OK) return st;
  if (n > 0 && C8 == nullptr) return BIGCN_EINVAL;
  if (!aligned(C8, 4)) return BIGCN_EALIGN;
  if (!bigcn::q8_supported(n, d, K) || (uint64_t)n * ldc8 > 0xFFFFFFFFull ||
      (uint64_t)n * ldc16 * 2 > 0xFFFFFFFFull)
    return BIGCN_EUNSUPPORTED;
  const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, d);
  if (n > 0 && nnz > 0) {
    if (workspace == nullptr || ws_bytes < plan.bytes) return BIGCN_EWORKSPACE;
    if (!aligned(workspace, 256)) return BIGCN_EALIGN;
  }
  hipStream_t s = (hipStream_t)stream;
  return hip_status(bigcn::launch_spmm_q8(n, nnz, rowptr, colidx, norm == BIGCN_NORM_MEAN,
                                          g, C8, ldc8, C16, ldc16, K, d, alpha, bias,
                                          act == BIGCN_ACT_RELU, out, ldo, plan,
                                          workspace, nullptr, s));
}

size_t bigcn_spmm_csr_q8_noalloc_max_bytes(void) { return kNoallocScratchBytes; }

bigcn_status bigcn_spmm_csr_q8_noalloc(int64_t n, int64_t nnz, const int64_t* rowptr,
                                       const int32_t* colidx, bigcn_norm norm,
                                       const float* g, const int8_t* C8, int64_t ldc8,
                                       const void* C16, int64_t ldc16, int32_t K,
                                       int32_t d, const float* alpha, const float* bias,
                                       bigcn_act act, float* out, int64_t ldo,
                                       void* stream) {
  bigcn_status st = check_graph(n, nnz, rowptr, colidx, norm);
  if (st != BIGCN_OK) return st;
  if (K < 1 || d < 1 || ldc8 < q8_row(d) || ldc8 % 4 != 0 || ldc16 < q8_row(d))
    return BIGCN_EINVAL;
  st = check_spmm_operands(n, g, C16, BIGCN_F16, d, ldc16, alpha, bias, act, out, ldo);
  if (st != BIGCN_OK) return st;
  if (n > 0 && C8 == nullptr) return BIGCN_EINVAL;
  if (!aligned(C8, 4)) return BIGCN_EALIGN;
  if (!bigcn::q8_supported(n, d, K) || (uint64_t)n * ldc8 > 0xFFFFFFFFull ||
      (uint64_t)n * ldc16 * 2 > 0xFFFFFFFFull)
    return BIGCN_EUNSUPPORTED;
  // Graphs of up to 67M entries get the plan bigcn_spmm_csr_q8 uses (the
  // same chunks, hence the same sums); larger ones wider chunks.
  const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, d, kNoallocWorkers);
  if (plan.bytes > kNoallocScratchBytes) return BIGCN_EWORKSPACE;
  void* ws = nullptr;
  if (n > 0 && nnz > 0) {
    ws = device_scratch();
    if (ws == nullptr) return BIGCN_EHIP;
  }
  return hip_status(bigcn::launch_spmm_q8(n, nnz, rowptr, colidx, norm == BIGCN_NORM_MEAN,
                                          g, C8, ldc8, C16, ldc16, K, d, alpha, bias,
                                          act == BIGCN_ACT_RELU, out, ldo, plan, ws, nullptr,
                                          (hipStream_t)stream));
}

bigcn_status bigcn_spmm_csr_sage_q8(int64_t n, int64_t nnz, const int64_t* rowptr,
                                    const int32_t* colidx, const float* g,
                                    const int8_t* C8, int64_t ldc8, const void* C16,
                                    int64_t ldc16, int32_t K, int32_t d,
                                    const float* alpha_neigh, const void* Cself,
                                    int64_t ldself, const float* alpha_self,
                                    const float* bias, bigcn_act act, float* out,
                                    int64_t ldo, void* workspace, size_t ws_bytes,
                                    void* stream) {
  bigcn_status st = check_graph(n, nnz, rowptr, colidx, BIGCN_NORM_MEAN);
  if (st != BIGCN_OK) return st;
  if (K < 1 || d < 1 || ldc8 < q8_row(d) || ldc8 % 4 != 0 || ldc16 < q8_row(d))
    return BIGCN_EINVAL;
  st = check_spmm_operands(n, g, C16, BIGCN_F16, d, ldc16, alpha_neigh, bias, act, out,
                           ldo);
  if (st != BIGCN_OK) return st;
  if (ldself < d || alpha_self == nullptr || (n > 0 && (C8 == nullptr || Cself == nullptr)))
    return BIGCN_EINVAL;
  if (!aligned(C8, 4) || !aligned(Cself, 2) || !aligned(alpha_self, 4)) return BIGCN_EALIGN;
  if (!bigcn::q8_supported(n, d, K) || (uint64_t)n * ldc8 > 0xFFFFFFFFull ||
      (uint64_t)n * ldc16 * 2 > 0xFFFFFFFFull)
    return BIGCN_EUNSUPPORTED;
  const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, d);
  if (n > 0 && nnz > 0) {
    if (workspace == nullptr || ws_bytes < plan.bytes) return BIGCN_EWORKSPACE;
    if (!aligned(workspace, 256)) return BIGCN_EALIGN;
  }
  bigcn::FusedNext fn = {};
  fn.kind = 2;
  fn.Cself = Cself;
  fn.ldself = ldself;
  fn.alpha_self = alpha_self;
  return hip_status(bigcn::launch_spmm_q8(n, nnz, rowptr, colidx, 1, g, C8, ldc8, C16, ldc16,
                                          K, d, alpha_neigh, bias, act == BIGCN_ACT_RELU,
                                          out, ldo, plan, workspace, &fn,
                                          (hipStream_t)stream));
}

size_t bigcn_source_slots_workspace_bytes(int64_t n) {
  if (n < 0) return 0;
  return bigcn::source_slots_plan(n).bytes;
}

bigcn_status bigcn_source_slots(int64_t n, int64_t nnz, const int64_t* rowptr,
                                const int32_t* colidx, int32_t* slot, int32_t* colslot,
                                void* workspace, size_t ws_bytes, void* stream) {
  if (n < 0 || nnz < 0 || n > INT32_MAX) return BIGCN_EINVAL;
  if (n > 0 && (rowptr == nullptr || slot == nullptr)) return BIGCN_EINVAL;
  if (nnz > 0 && (colidx == nullptr || colslot == nullptr)) return BIGCN_EINVAL;
  if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(slot, 4) || !aligned(colslot, 4))
    return BIGCN_EALIGN;
  if (n == 0) return BIGCN_OK;
  if (workspace == nullptr || ws_bytes < bigcn::source_slots_plan(n).bytes)
    return BIGCN_EWORKSPACE;
  if (!aligned(workspace, 256)) return BIGCN_EALIGN;
  return hip_status(bigcn::launch_source_slots(n, nnz, rowptr, colidx, slot, colslot,
                                               workspace, (hipStream_t)stream));
}

size_t bigcn_forward_workspace_bytes(int64_t n, int64_t nnz,
                                     const bigcn_layer* layers, int32_t n_layers) {
  if (n < 0 || nnz < 0 || layers == nullptr || n_layers < 1) return 0;
  for (int32_t l = 0; l < n_layers; ++l)
    if (layers[l].d_in < 1 || layers[l].d_out < 1) return 0;
  ForwardLayout L;
  forward_layout(n, nnz, layers, n_layers, &L);
  return L.bytes;
}

bigcn_status bigcn_forward(int64_t n, int64_t nnz, const int64_t* rowptr,
                           const int32_t* colidx, const int32_t* slot,
                           const int32_t* colslot, bigcn_norm norm,
                           const float* x, int64_t ldx, const float* mu,
                           const float* rstd, const bigcn_layer* layers,
                           int32_t n_layers, float* out, int64_t ldo,
                           void* workspace, size_t ws_bytes, void* stream) {
  if (layers == nullptr || n_layers < 1) return BIGCN_EINVAL;
  bigcn_status st = check_graph(n, nnz, rowptr, colidx, norm);
  if (st != BIGCN_OK) return st;
  if ((slot == nullptr) != (colslot == nullptr)) return BIGCN_EINVAL;
  if (!aligned(slot, 4) || !aligned(colslot, 4)) return BIGCN_EALIGN;
  if (nnz == 0) {  // nothing is gathered: any order is the same
    slot = nullptr;
    colslot = nullptr;
  }
  // the aggregations gather sources by slot when a source order is given
  const int32_t* gcol = colslot != nullptr ? colslot : colidx;
  for (int32_t l = 0; l < n_layers; ++l) {
    const bigcn_layer& ly = layers[l];
    if (ly.d_in < 1 || ly.d_out < 1 || ly.ldw < words(ly.d_in)) return BIGCN_EINVAL;
    if (l > 0 && ly.d_in != layers[l - 1].d_out) return BIGCN_EINVAL;
    if (ly.wbits == nullptr || ly.alpha == nullptr) return BIGCN_EINVAL;
    if (ly.act != BIGCN_ACT_NONE && ly.act != BIGCN_ACT_RELU) return BIGCN_EINVAL;
    if (!aligned(ly.wbits, 8) || !aligned(ly.alpha, 4) || !aligned(ly.bias, 4))
      return BIGCN_EALIGN;
    if (ly.d_in > kMaxBgemmK) return BIGCN_EUNSUPPORTED;
    if (l + 1 < n_layers && ly.out != nullptr) {  // a requested hidden output
      if (ly.ldo < ly.d_out) return BIGCN_EINVAL;
      if (!aligned(ly.out, 4)) return BIGCN_EALIGN;
    }
    if (ly.wbits_self != nullptr) {  // two-weight GraphSAGE layer
      if (ly.alpha_self == nullptr || ly.ldw_self < words(ly.d_in)) return BIGCN_EINVAL;
      if (!aligned(ly.wbits_self, 8) || !aligned(ly.alpha_self, 4)) return BIGCN_EALIGN;
      if (norm != BIGCN_NORM_MEAN) return BIGCN_EINVAL;
      if (!bigcn::q8_supported(n, ly.d_out, ly.d_in)) return BIGCN_EUNSUPPORTED;
    }
  }
  if (ldx < layers[0].d_in || ldo < layers[n_layers - 1].d_out) return BIGCN_EINVAL;
  if ((mu == nullptr) != (rstd == nullptr)) return BIGCN_EINVAL;
  if (n > 0 && (x == nullptr || out == nullptr)) return BIGCN_EINVAL;
  if (!aligned(x, 4) || !aligned(out, 4) || !aligned(mu, 4) || !aligned(rstd, 4))
    return BIGCN_EALIGN;
  ForwardLayout L;
  forward_layout(n, nnz, layers, n_layers, &L);
  if (n == 0) return BIGCN_OK;
  if (workspace == nullptr || ws_bytes < L.bytes) return BIGCN_EWORKSPACE;
  if (!aligned(workspace, 256)) return BIGCN_EALIGN;

  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  uint64_t* F = (uint64_t*)(ws + L.off_F);
  float* H[2] = {(float*)(ws + L.off_H0), (float*)(ws + L.off_H1)};
  void* wsp = ws + L.off_spmm;

  // The exact-product aggregation needs per-worker start rows; they depend
  // only on the graph and the chunk size (the same for every layer).  The
  // 8-bit aggregation finds its rows itself.
  hipError_t e = hipSuccess;
  bool need_rows = false;
  for (int32_t l = 0; l < n_layers; ++l)
    need_rows |= !bigcn::q8_supported(n, layers[l].d_out, layers[l].d_in);
  if (need_rows) {
    const bigcn::SpmmPlan plan0 = bigcn::spmm_plan(n, nnz, L.dmax);
    e = bigcn::launch_spmm_rows(n, nnz, rowptr, plan0, wsp, s);
    if (e != hipSuccess) return BIGCN_EHIP;
  }

  const float* hin = x;
  int64_t ldin = ldx;
  bool have_products = false;  // layer l's products already written by layer l-1
  for (int32_t l = 0; l < n_layers; ++l) {
    const bigcn_layer& ly = layers[l];
    const bool last = l + 1 == n_layers;
    const int set = l & 1;
    float* g = (float*)(ws + L.off_g[set]);
    int8_t* C8 = (int8_t*)(ws + L.off_C8[set]);
    void* C16 = ws + L.off_C16[set];
    const bool q8 = bigcn::q8_supported(n, ly.d_out, ly.d_in);
    const IType ct = forward_itype(ly.d_in);
    if (!have_products && q8 && ly.wbits_self == nullptr &&
        bigcn::pack_bgemm_q8_supported(ly.d_in, ly.d_out, ldin)) {
      e = bigcn::launch_pack_bgemm_q8(hin, n, ly.d_in, ldin, l == 0 ? mu : nullptr,
                                      l == 0 ? rstd : nullptr, rowptr,
                                      norm == BIGCN_NORM_SYM, ly.wbits, ly.d_out, ly.ldw,
                                      C8, q8_row(ly.d_out), C16, q8_row(ly.d_out), g, s,
                                      slot);
      if (e != hipSuccess) return BIGCN_EHIP;
    } else if (!have_products) {
      e = bigcn::launch_pack(hin, n, ly.d_in, ldin, l == 0 ? mu : nullptr,
                             l == 0 ? rstd : nullptr, rowptr, norm == BIGCN_NORM_SYM,
                             F, L.ldF, g, s, slot);
      if (e != hipSuccess) return BIGCN_EHIP;
      if (q8)
        e = bigcn::launch_bgemm_q8(F, n, L.ldF, ly.wbits, ly.d_out, ly.ldw, ly.d_in, C8,
                                   q8_row(ly.d_out), C16, q8_row(ly.d_out), g, s);
      else
        e = run_bgemm(F, n, L.ldF, ly.wbits, ly.d_out, ly.ldw, ly.d_in, C16, ct, L.ldc16,
                      BIGCN_BGEMM_AUTO, s);
      if (e != hipSuccess) return BIGCN_EHIP;
      // the node's own products, exact in half, unless the aggregation forms
      // them in its epilogue from F
      if (ly.wbits_self != nullptr &&
          !bigcn::self_in_epilogue_supported(nnz, ly.d_out, ly.d_in)) {
        e = run_bgemm(F, n, L.ldF, ly.wbits_self, ly.d_out, ly.ldw_self, ly.d_in,
                      ws + L.off_S, IType::F16, L.ldS, BIGCN_BGEMM_AUTO, s);
        if (e != hipSuccess) return BIGCN_EHIP;
      }
    }
    const int kind = fuse_kind(n, nnz, layers, n_layers, l);
    // the layer's fp32 output: the caller's for the last layer or when asked
    // for, else the workspace (none when the epilogue forms the next layer's
    // products)
    float* hout = last ? out
                       : (ly.out != nullptr ? ly.out : (kind != 0 ? nullptr : H[l & 1]));
    const int64_t ldout = last ? ldo : (ly.out != nullptr ? ly.ldo : L.ldh);
    const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, ly.d_out);
    if (q8) {
      bigcn::FusedNext fn = {};
      fn.kind = kind;
      fn.slot = slot;
      if (ly.wbits_self != nullptr) {
        fn.alpha_self = ly.alpha_self;
        if (bigcn::self_in_epilogue_supported(nnz, ly.d_out, ly.d_in)) {
          fn.kind = 3;
          fn.F = F;
          fn.ldF = L.ldF;
          fn.wself = ly.wbits_self;
          fn.ldw_self = ly.ldw_self;
          fn.kin = ly.d_in;
        } else {
          fn.kind = 2;
          fn.Cself = ws + L.off_S;
          fn.ldself = L.ldS;
        }
      } else if (kind != 0) {
        const bigcn_layer& nxt = layers[l + 1];
        const int nset = (l + 1) & 1;
        fn.wbits = nxt.wbits;
        fn.ldw = nxt.ldw;
        fn.d_out = nxt.d_out;
        fn.C8 = (int8_t*)(ws + L.off_C8[nset]);
        fn.ldc8 = q8_row(nxt.d_out);
        fn.C16 = ws + L.off_C16[nset];
        fn.ldc16 = q8_row(nxt.d_out);
        fn.g = (float*)(ws + L.off_g[nset]);
      }
      e = bigcn::launch_spmm_q8(n, nnz, rowptr, gcol, norm == BIGCN_NORM_MEAN, g, C8,
                                q8_row(ly.d_out), C16, q8_row(ly.d_out), ly.d_in, ly.d_out,
                                ly.alpha, ly.bias,
                                ly.act == BIGCN_ACT_RELU, hout, ldout, plan, wsp, &fn, s);
    } else {
      e = bigcn::launch_spmm(n, nnz, rowptr, gcol, norm == BIGCN_NORM_MEAN, g, C16, ct,
                             ly.d_out, L.ldc16, ly.alpha, ly.bias, ly.act == BIGCN_ACT_RELU,
                             hout, ldout, plan, wsp, s);
    }
    if (e != hipSuccess) return BIGCN_EHIP;
    have_products = kind != 0;
    hin = hout;
    ldin = ldout;
  }
  return BIGCN_OK;
}

}  // extern "C"
