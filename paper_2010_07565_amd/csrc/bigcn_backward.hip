// Back propagation of one binarized graph-convolution layer on gfx950
// (Alg. 1 with Eqs. (14)-(15)): the gradients of the binarized weights and
// features, the straight-through weight gradient, and the gradient passed to
// the layer below.  C ABI entry points at the end of the file.
//
// Steps (G = dL/dH^(l+1), masked by the ReLU when the layer has one):
//   db    = column sums of G                     (fixed-order, fp64 partials)
//   dζ    = Ã^T G                                (the edge-chunked aggregation
//                                                 of bigcn_kernels.hip on fp32
//                                                 rows; Â structurally symmetric)
//   dW~^T = (H~^T dζ)^T,  H~ = diag(β) F         (fp64 partial sums per chunk
//                                                 of rows, summed in order)
//   dH~   = dζ W~^T,      W~ = B diag(α);  dH = dH~ 1[|dH~| < 1]   (Eq. (14))
//   dW    = Eq. (15) with 1[|W| < 1] for the derivative of sign.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/bigcn.h"
#include "bigcn_internal.h"

namespace {

constexpr int kB = 256;  // threads per block (4 waves)

inline size_t up256(size_t v) { return (v + 255) & ~(size_t)255; }
inline int64_t words(int64_t k) { return (k + 63) / 64; }

// Gm = G (zero where the ReLU output is not positive, and in the pad columns
// up to ldm); s_i = the source-side factor of Ã^T (D̂_ii^-1/2 symmetric,
// D̂_ii^-1 mean); ones = 1 (the per-column scale of the aggregation).
__global__ __launch_bounds__(kB) void k_bwd_prep(
    int64_t n, int32_t d, const float* __restrict__ G, int64_t ldg,
    const float* __restrict__ out, int64_t ldo, int relu, float* __restrict__ Gm,
    int64_t ldm, const int64_t* __restrict__ rowptr, int mean, float* __restrict__ s,
    float* __restrict__ ones) {
  const int64_t idx = (int64_t)blockIdx.x * kB + threadIdx.x;
  if (idx < n * ldm) {
    const int64_t i = idx / ldm;
    const int64_t k = idx - i * ldm;
    float v = 0.f;
    if (k < d) {
      v = G[i * ldg + k];
      if (relu && !(out[i * ldo + k] > 0.f)) v = 0.f;
    }
    Gm[idx] = v;
  }
  if (idx < n) {
    const int64_t deg = rowptr[idx + 1] - rowptr[idx];
    const float dg = (float)deg;
    s[idx] = deg > 0 ? (mean ? 1.0f / dg : 1.0f / sqrtf(dg)) : 0.f;
  }
  if (idx < d) ones[idx] = 1.f;
}

// Column sums of Gm over a chunk of R rows (block = chunk), fp64, rows in
// order (eight loads in flight); then the chunks in order.
__global__ __launch_bounds__(kB) void k_bwd_colsum_part(
    int64_t n, int32_t d, const float* __restrict__ Gm, int64_t ldm, int64_t R,
    double* __restrict__ part) {
  const int64_t c = blockIdx.x;
  const int64_t i0 = c * R, i1 = std::min<int64_t>(n, i0 + R);
  for (int k = threadIdx.x; k < d; k += kB) {
    double acc = 0.0;
    int64_t i = i0;
    for (; i + 8 <= i1; i += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = Gm[(i + u) * ldm + k];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += (double)v[u];
    }
    for (; i < i1; ++i) acc += (double)Gm[i * ldm + k];
    part[c * d + k] = acc;
  }
}

__global__ __launch_bounds__(kB) void k_bwd_colsum_final(
    int32_t d, int64_t chunks, const double* __restrict__ part, float* __restrict__ db) {
  const int k = blockIdx.x * kB + threadIdx.x;
  if (k >= d) return;
  double acc = 0.0;
  int64_t c = 0;
  for (; c + 8 <= chunks; c += 8) {  // eight loads in flight, added in order
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = part[(c + u) * d + k];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; c < chunks; ++c) acc += part[c * d + k];
  db[k] = (float)acc;
}

// Partial sums of dW~^T over a chunk of R rows:
//   part[c][j][64w + b] = sum_{i in chunk c} s(F_i, 64w + b) * β_i dζ_ij.
// Block (chunk c, word w, 64 columns): thread (column j, bit group q) owns
// bits 16q .. 16q+15 of the word for column j.  Each run of 64 rows is
// summed in fp32 (at most 64 terms) and added to fp64 accumulators, in row
// order.  Row words are wave-uniform.
__global__ __launch_bounds__(kB) void k_bwd_wtilde_part(
    int64_t n, int32_t d_in, int32_t d_out, const uint64_t* __restrict__ F, int64_t ldf,
    const float* __restrict__ beta, const float* __restrict__ dz, int64_t lddz,
    int64_t R, double* __restrict__ part) {
  const int64_t c = blockIdx.x;
  const int w = blockIdx.y;
  const int j = blockIdx.z * 64 + (threadIdx.x & 63);
  const int q = threadIdx.x >> 6;  // wave index: bit group
  if (j >= d_out) return;          // no barrier in this kernel
  const int64_t i0 = c * R, i1 = std::min<int64_t>(n, i0 + R);
  double acc[16];
#pragma unroll
  for (int b = 0; b < 16; ++b) acc[b] = 0.0;
  for (int64_t r0 = i0; r0 < i1; r0 += 64) {
    const int64_t r1 = std::min<int64_t>(i1, r0 + 64);
    float sub[16];
#pragma unroll
    for (int b = 0; b < 16; ++b) sub[b] = 0.f;
    int64_t i = r0;
    for (; i + 8 <= r1; i += 8) {  // eight rows' loads in flight, summed in order
      float x[8];
      uint32_t bits[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        x[u] = beta[i + u] * dz[(i + u) * lddz + j];
        bits[u] = (uint32_t)(F[(i + u) * ldf + w] >> (16 * q)) & 0xFFFFu;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int b = 0; b < 16; ++b) sub[b] += ((bits[u] >> b) & 1u) ? x[u] : -x[u];
    }
    for (; i < r1; ++i) {
      const float x = beta[i] * dz[i * lddz + j];
      const uint32_t bits = (uint32_t)(F[i * ldf + w] >> (16 * q)) & 0xFFFFu;
#pragma unroll
      for (int b = 0; b < 16; ++b) sub[b] += ((bits >> b) & 1u) ? x : -x;
    }
#pragma unroll
    for (int b = 0; b < 16; ++b) acc[b] += (double)sub[b];
  }
  double* dst = part + ((int64_t)c * d_out + j) * d_in + 64 * w + 16 * q;
  const int nb = std::min(16, d_in - 64 * w - 16 * q);
#pragma unroll
  for (int b = 0; b < 16; ++b)
    if (b < nb) dst[b] = acc[b];
}

// dW~^T[j][k] = sum over chunks in order; fp64 kept for Eq. (15), fp32 copy
// to the caller (optional).
__global__ __launch_bounds__(kB) void k_bwd_wtilde_final(
    int32_t d_in, int32_t d_out, int64_t chunks, const double* __restrict__ part,
    double* __restrict__ wtd, float* __restrict__ out, int64_t ldout) {
  const int64_t idx = (int64_t)blockIdx.x * kB + threadIdx.x;
  if (idx >= (int64_t)d_in * d_out) return;
  const int64_t j = idx / d_in, k = idx - j * d_in;
  double acc = 0.0;
  int64_t c = 0;
  for (; c + 8 <= chunks; c += 8) {  // eight loads in flight, added in order
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = part[((c + u) * d_out + j) * d_in + k];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; c < chunks; ++c) acc += part[(c * d_out + j) * d_in + k];
  wtd[idx] = acc;
  if (out != nullptr) out[j * ldout + k] = (float)acc;
}

// Eq. (15) for column j of W (row j of W^T), block j:
//   dW_ij = B_ij / d_in * sum_k dW~_kj B_kj + α_j dW~_ij 1[|W_ij| < 1].
__global__ __launch_bounds__(kB) void k_bwd_weights(
    int32_t d_in, const double* __restrict__ wtd, const uint64_t* __restrict__ B,
    int64_t ldb, const float* __restrict__ alpha, const float* __restrict__ wt,
    int64_t ldwt, float* __restrict__ dwt, int64_t lddw) {
  __shared__ double red[kB];
  const int j = blockIdx.x;
  const uint64_t* bj = B + (int64_t)j * ldb;
  const double* g = wtd + (int64_t)j * d_in;
  double acc = 0.0;
  for (int k = threadIdx.x; k < d_in; k += kB)
    acc += ((bj[k >> 6] >> (k & 63)) & 1ull) ? g[k] : -g[k];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int off = kB / 2; off > 0; off >>= 1) {  // fixed-order tree
    if ((int)threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  const double colsum = red[0];
  const double a = (double)alpha[j];
  for (int i = threadIdx.x; i < d_in; i += kB) {
    const double bij = ((bj[i >> 6] >> (i & 63)) & 1ull) ? 1.0 : -1.0;
    const double ste = fabsf(wt[(int64_t)j * ldwt + i]) < 1.0f ? 1.0 : 0.0;
    dwt[(int64_t)j * lddw + i] = (float)(bij * colsum / (double)d_in + a * g[i] * ste);
  }
}

// dH~[i][k] = sum_j dζ_ij α_j s(B_j, k), j in order, and Eq. (14).  One
// wave per row; lane l owns columns 64w + l (w < kw <= KW); the packed
// weight words sit in LDS ([d_out][kw]) and are read as wave broadcasts.
template <int KW>
__global__ __launch_bounds__(kB) void k_bwd_htilde(
    int64_t n, int32_t d_in, int32_t d_out, const float* __restrict__ dz, int64_t lddz,
    const uint64_t* __restrict__ B, int64_t ldb, const float* __restrict__ alpha,
    float* __restrict__ dht, int64_t lddht, float* __restrict__ dh, int64_t lddh) {
  extern __shared__ uint64_t sB[];
  const int kw = (d_in + 63) >> 6;
  for (int idx = threadIdx.x; idx < d_out * kw; idx += kB)
    sB[idx] = B[(int64_t)(idx / kw) * ldb + idx % kw];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * (kB / 64);
  for (int64_t i = (int64_t)blockIdx.x * (kB / 64) +
                   __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
       i < n; i += nwaves) {
    float acc[KW];
#pragma unroll
    for (int w = 0; w < KW; ++w) acc[w] = 0.f;
    for (int j0 = 0; j0 < d_out; j0 += 64) {
      const int jl = j0 + lane;
      const float v = jl < d_out ? alpha[jl] * dz[i * lddz + jl] : 0.f;
      const int jn = std::min(64, d_out - j0);
      for (int jj = 0; jj < jn; ++jj) {
        const float vj = __builtin_bit_cast(
            float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), jj));
        const uint64_t* row = sB + (j0 + jj) * kw;
#pragma unroll
        for (int w = 0; w < KW; ++w) {
          if (w >= kw) break;
          acc[w] += ((row[w] >> lane) & 1ull) ? vj : -vj;
        }
      }
    }
#pragma unroll
    for (int w = 0; w < KW; ++w) {
      const int k = 64 * w + lane;
      if (w >= kw || k >= d_in) break;
      if (dht != nullptr) dht[i * lddht + k] = acc[w];
      if (dh != nullptr) dh[i * lddh + k] = fabsf(acc[w]) < 1.f ? acc[w] : 0.f;
    }
  }
}

inline unsigned grid_of(int64_t threads) {
  return (unsigned)std::max<int64_t>(1, (threads + kB - 1) / kB);
}

// Workspace layout of bigcn_layer_backward.
struct BwdLayout {
  int64_t kw, ldm, R, chunks, Rdb, chunks_db;
  size_t off_F, off_beta, off_s, off_ones, off_Gm, off_dz, off_pdb, off_pw, off_wtd,
      off_spmm, bytes;
};

BwdLayout bwd_layout(int64_t n, int64_t nnz, int32_t d_in, int32_t d_out) {
  BwdLayout L;
  L.kw = words(d_in);
  L.ldm = (d_out + 3) / 4 * 4;
  // Row chunks of the dW~ partial sums: about 2048 blocks of (chunk, word,
  // 64 columns), chunks of at least 64 rows, partial sums within 512 MB.
  const int64_t per_chunk = L.kw * ((d_out + 63) / 64);
  int64_t chunks = std::max<int64_t>(1, 2048 / per_chunk);
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (n + 63) / 64));
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (512ll << 20) / ((int64_t)d_out * d_in * 8)));
  L.R = std::max<int64_t>(1, (n + chunks - 1) / chunks);
  L.chunks = std::max<int64_t>(1, (n + L.R - 1) / L.R);
  L.Rdb = std::max<int64_t>(64, (n + 4095) / 4096);  // at most 4096 row chunks
  L.chunks_db = std::max<int64_t>(1, (n + L.Rdb - 1) / L.Rdb);
  size_t off = 0;
  L.off_F = off;
  off += up256((size_t)n * L.kw * 8);
  L.off_beta = off;
  off += up256((size_t)n * 4);
  L.off_s = off;
  off += up256((size_t)n * 4);
  L.off_ones = off;
  off += up256((size_t)L.ldm * 4);
  L.off_Gm = off;
  off += up256((size_t)n * L.ldm * 4);
  L.off_dz = off;
  off += up256((size_t)n * L.ldm * 4);
  L.off_pdb = off;
  off += up256((size_t)L.chunks_db * d_out * 8);
  L.off_pw = off;
  off += up256((size_t)L.chunks * d_out * d_in * 8);
  L.off_wtd = off;
  off += up256((size_t)d_out * d_in * 8);
  L.off_spmm = off;
  off += bigcn::spmm_plan(n, nnz, d_out).bytes;
  L.bytes = off;
  return L;
}

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

template <int KW>
void launch_htilde(int64_t n, int32_t d_in, int32_t d_out, const float* dz, int64_t lddz,
                   const uint64_t* B, int64_t ldb, const float* alpha, float* dht,
                   int64_t lddht, float* dh, int64_t lddh, hipStream_t s) {
  const size_t lds = (size_t)d_out * words(d_in) * 8;
  const int64_t blocks = std::min<int64_t>((n + 3) / 4, 8192);
  hipLaunchKernelGGL((k_bwd_htilde<KW>), dim3((unsigned)std::max<int64_t>(1, blocks)),
                     dim3(kB), lds, s, n, d_in, d_out, dz, lddz, B, ldb, alpha, dht, lddht,
                     dh, lddh);
}

}  // namespace

extern "C" {

size_t bigcn_layer_backward_workspace_bytes(int64_t n, int64_t nnz, int32_t d_in,
                                            int32_t d_out) {
  if (n < 0 || nnz < 0 || d_in < 1 || d_out < 1) return 0;
  return bwd_layout(n, nnz, d_in, d_out).bytes;
}

bigcn_status bigcn_layer_backward(int64_t n, int64_t nnz, const int64_t* rowptr,
                                  const int32_t* colidx, bigcn_norm norm, const float* h,
                                  int64_t ldh, int32_t d_in, const float* wt, int64_t ldwt,
                                  const uint64_t* wbits, int64_t ldw, const float* alpha,
                                  int32_t d_out, const float* gout, int64_t ldg,
                                  const float* out, int64_t ldo, bigcn_act act,
                                  float* dh, int64_t lddh, float* dh_tilde,
                                  int64_t lddht, float* dwt, int64_t lddw,
                                  float* dwt_tilde, int64_t lddwt, float* db,
                                  float* dzeta, int64_t lddz, void* workspace,
                                  size_t ws_bytes, void* stream) {
  if (n < 0 || nnz < 0 || n > INT32_MAX || d_in < 1 || d_in > 2048 || d_out < 1 ||
      d_out > 256)
    return d_in > 2048 || d_out > 256 ? BIGCN_EUNSUPPORTED : BIGCN_EINVAL;
  if (norm != BIGCN_NORM_SYM && norm != BIGCN_NORM_MEAN) return BIGCN_EINVAL;
  if (act != BIGCN_ACT_NONE && act != BIGCN_ACT_RELU) return BIGCN_EINVAL;
  if (ldh < d_in || ldwt < d_in || ldw < words(d_in) || ldg < d_out) return BIGCN_EINVAL;
  if (wt == nullptr || wbits == nullptr || alpha == nullptr || dwt == nullptr ||
      lddw < d_in)
    return BIGCN_EINVAL;
  if (n > 0 && (rowptr == nullptr || h == nullptr || gout == nullptr)) return BIGCN_EINVAL;
  if (nnz > 0 && colidx == nullptr) return BIGCN_EINVAL;
  if (act == BIGCN_ACT_RELU && n > 0 && (out == nullptr || ldo < d_out)) return BIGCN_EINVAL;
  if ((dh != nullptr && lddh < d_in) || (dh_tilde != nullptr && lddht < d_in) ||
      (dwt_tilde != nullptr && lddwt < d_in) || (dzeta != nullptr && lddz < d_out))
    return BIGCN_EINVAL;
  if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(h, 4) || !aligned(wt, 4) ||
      !aligned(wbits, 8) || !aligned(alpha, 4) || !aligned(gout, 4) || !aligned(out, 4) ||
      !aligned(dh, 4) || !aligned(dh_tilde, 4) || !aligned(dwt, 4) ||
      !aligned(dwt_tilde, 4) || !aligned(db, 4) || !aligned(dzeta, 4))
    return BIGCN_EALIGN;
  const BwdLayout L = bwd_layout(n, nnz, d_in, d_out);
  if (workspace == nullptr || ws_bytes < L.bytes) return BIGCN_EWORKSPACE;
  if (!aligned(workspace, 256)) return BIGCN_EALIGN;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  uint64_t* F = (uint64_t*)(ws + L.off_F);
  float* beta = (float*)(ws + L.off_beta);
  float* sc = (float*)(ws + L.off_s);
  float* ones = (float*)(ws + L.off_ones);
  float* Gm = (float*)(ws + L.off_Gm);
  float* dz = (float*)(ws + L.off_dz);
  double* pdb = (double*)(ws + L.off_pdb);
  double* pw = (double*)(ws + L.off_pw);
  double* wtd = (double*)(ws + L.off_wtd);
  void* wsp = ws + L.off_spmm;
  const int mean = norm == BIGCN_NORM_MEAN;
  hipError_t e;
#define BIGCN_CHECK(x)                      \
  do {                                      \
    e = (x);                                \
    if (e != hipSuccess) return BIGCN_EHIP; \
  } while (0)

  // Signs and β of the layer input (Eqs. (7)-(8); no normalisation factor).
  if (n > 0)
    BIGCN_CHECK(bigcn::launch_pack(h, n, d_in, ldh, nullptr, nullptr, nullptr, 0, F, L.kw,
                                   beta, s));
  hipLaunchKernelGGL(k_bwd_prep, dim3(grid_of(std::max<int64_t>(n * L.ldm, L.ldm))),
                     dim3(kB), 0, s, n, d_out, gout, ldg, out, ldo,
                     act == BIGCN_ACT_RELU ? 1 : 0, Gm, L.ldm, rowptr, mean, sc, ones);
  BIGCN_CHECK(hipGetLastError());
  if (db != nullptr) {
    hipLaunchKernelGGL(k_bwd_colsum_part, dim3((unsigned)L.chunks_db), dim3(kB), 0, s, n,
                       d_out, Gm, L.ldm, L.Rdb, pdb);
    hipLaunchKernelGGL(k_bwd_colsum_final, dim3(grid_of(d_out)), dim3(kB), 0, s, d_out,
                       L.chunks_db, pdb, db);
    BIGCN_CHECK(hipGetLastError());
  }
  // dζ = Ã^T G: sources scaled by s_i, destinations by D̂^-1/2 (symmetric)
  // or not at all (mean, normalisation mode 2).
  if (n > 0) {
    const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, d_out);
    BIGCN_CHECK(bigcn::launch_spmm_rows(n, nnz, rowptr, plan, wsp, s));
    BIGCN_CHECK(bigcn::launch_spmm(n, nnz, rowptr, colidx, mean ? 2 : 0, sc, Gm,
                                   bigcn::IType::F32, d_out, L.ldm, ones, nullptr, 0, dz,
                                   L.ldm, plan, wsp, s));
    if (dzeta != nullptr)
      BIGCN_CHECK(hipMemcpy2DAsync(dzeta, lddz * 4, dz, L.ldm * 4, (size_t)d_out * 4, n,
                                   hipMemcpyDeviceToDevice, s));
  }
  // dW~^T, then Eq. (15).
  hipLaunchKernelGGL(k_bwd_wtilde_part, dim3((unsigned)L.chunks, (unsigned)L.kw,
                                             (unsigned)((d_out + 63) / 64)),
                     dim3(kB), 0, s, n, d_in, d_out, F, L.kw, beta, dz, L.ldm, L.R, pw);
  hipLaunchKernelGGL(k_bwd_wtilde_final, dim3(grid_of((int64_t)d_in * d_out)), dim3(kB), 0,
                     s, d_in, d_out, L.chunks, pw, wtd, dwt_tilde, lddwt);
  hipLaunchKernelGGL(k_bwd_weights, dim3((unsigned)d_out), dim3(kB), 0, s, d_in, wtd, wbits,
                     ldw, alpha, wt, ldwt, dwt, lddw);
  BIGCN_CHECK(hipGetLastError());
  // dH~ and dH (Eq. (14)).
  if (n > 0 && (dh != nullptr || dh_tilde != nullptr)) {
    const int kw = (int)L.kw;
#define BIGCN_HT(KWV)                                                                     \
  launch_htilde<KWV>(n, d_in, d_out, dz, L.ldm, wbits, ldw, alpha, dh_tilde, lddht, dh, \
                     lddh, s)
    if (kw <= 1) BIGCN_HT(1);
    else if (kw <= 2) BIGCN_HT(2);
    else if (kw <= 4) BIGCN_HT(4);
    else if (kw <= 8) BIGCN_HT(8);
    else if (kw <= 16) BIGCN_HT(16);
    else BIGCN_HT(32);
#undef BIGCN_HT
    BIGCN_CHECK(hipGetLastError());
  }
#undef BIGCN_CHECK
  return BIGCN_OK;
}

}  // extern "C"
