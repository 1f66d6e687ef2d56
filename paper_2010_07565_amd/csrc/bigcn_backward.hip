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
//   dW~^T = (H~^T dζ)^T,  H~ = diag(β) F         (bf16 MFMA on the exact
//                                                 three-piece split of the fp32
//                                                 operand; 64-row runs added to
//                                                 fp64 partial sums per chunk of
//                                                 rows, summed in order)
//   dH~   = dζ W~^T,      W~ = B diag(α);  dH = dH~ 1[|dH~| < 1]   (Eq. (14);
//                                                 bf16 MFMA, the same split)
//   dW    = Eq. (15) with 1[|W| < 1] for the derivative of sign.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/bigcn.h"
#include "bigcn_internal.h"

namespace {

constexpr int kB = 256;  // threads per block (4 waves)
typedef float float4_t __attribute__((ext_vector_type(4)));

inline size_t up256(size_t v) { return (v + 255) & ~(size_t)255; }
inline int64_t words(int64_t k) { return (k + 63) / 64; }

// Gm = G (zero where the ReLU output is not positive, and in the pad columns
// up to ldm), unless Gm is null (G is then aggregated in place); s_i = the
// source-side factor of Ã^T (D̂_ii^-1/2 symmetric, D̂_ii^-1 mean); ones = 1
// (the per-column scale of the aggregation).  With slot, node i's row of Gm
// and its factor go to position slot[i] (the source order of the forward
// pass), where the aggregation reads them through the column slots.
// A row takes 2^lpr_log2 lanes (the power of two covering ldm / 4 quads,
// ldm <= 256 a multiple of 4), so a wave stages 64 >> lpr_log2 rows; lane
// quad c covers columns 4c .. 4c+3 with one 16-byte store (Gm 16-byte
// aligned), reading G (and out) as one 16-byte load each when vec (d and
// their row strides multiples of 4, both 16-byte aligned).
__global__ __launch_bounds__(kB) void k_bwd_prep(
    int64_t n, int32_t d, const float* __restrict__ G, int64_t ldg,
    const float* __restrict__ out, int64_t ldo, int relu, float* __restrict__ Gm,
    int64_t ldm, const int64_t* __restrict__ rowptr, int mean, float* __restrict__ s,
    float* __restrict__ ones, const int32_t* __restrict__ slot, int lpr_log2, int vec) {
  const int lane = threadIdx.x & 63;
  const int64_t i = ((int64_t)blockIdx.x * (kB / 64) + (threadIdx.x >> 6)) * (64 >> lpr_log2) +
                    (lane >> lpr_log2);
  const int c = lane & ((1 << lpr_log2) - 1);
  if (i < n) {
    const int64_t dst = slot != nullptr ? (int64_t)slot[i] : i;
    if (Gm != nullptr && 4 * c < ldm) {
      float4_t v = {0.f, 0.f, 0.f, 0.f};
      if (vec) {
        v = *reinterpret_cast<const float4_t*>(G + i * ldg + 4 * c);
        float4_t o = {1.f, 1.f, 1.f, 1.f};
        if (relu) o = *reinterpret_cast<const float4_t*>(out + i * ldo + 4 * c);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (relu && !(o[u] > 0.f)) v[u] = 0.f;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int k = 4 * c + u;
          if (k < d) {
            const float x = G[i * ldg + k];
            v[u] = relu && !(out[i * ldo + k] > 0.f) ? 0.f : x;
          }
        }
      }
      *reinterpret_cast<float4_t*>(Gm + dst * ldm + 4 * c) = v;
    }
    if (c == 0) {
      const int64_t deg = rowptr[i + 1] - rowptr[i];
      const float dg = (float)deg;
      s[dst] = deg > 0 ? (mean ? 1.0f / dg : 1.0f / sqrtf(dg)) : 0.f;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < d) ones[threadIdx.x] = 1.f;
}

// Column sums of Gm over a chunk of R rows (block = chunk), fp64, rows in
// node order (row i at slot[i] when given; eight loads in flight); then the
// chunks in order.
__global__ __launch_bounds__(kB) void k_bwd_colsum_part(
    int64_t n, int32_t d, const float* __restrict__ Gm, int64_t ldm, int64_t R,
    double* __restrict__ part, const int32_t* __restrict__ slot) {
  const int64_t c = blockIdx.x;
  const int64_t i0 = c * R, i1 = std::min<int64_t>(n, i0 + R);
  auto row = [&](int64_t i) -> int64_t { return slot != nullptr ? (int64_t)slot[i] : i; };
  for (int k = threadIdx.x; k < d; k += kB) {
    double acc = 0.0;
    int64_t i = i0;
    for (; i + 8 <= i1; i += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = Gm[row(i + u) * ldm + k];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += (double)v[u];
    }
    for (; i < i1; ++i) acc += (double)Gm[row(i) * ldm + k];
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

// bf16 operands of the 16x16x32 matrix-core product: lane (m, q) holds eight
// consecutive K entries 8q .. 8q+7 of its A row m / B column m.
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16v2_t __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to nearest bf16 and packed, and those two bf16
// values back in fp32 (the packed halves moved into place).
__device__ inline uint32_t pk_bf16(float a, float b, float& fa, float& fb) {
  const f32x2_t v = {a, b};
  const uint32_t p = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16v2_t));
  fa = __builtin_bit_cast(float, p << 16);
  fb = __builtin_bit_cast(float, p & 0xFFFF0000u);
  return p;
}

// x = h + md + lo exactly for normal fp32 x: each piece is the remainder of
// the previous ones rounded to bf16 (8 significant bits each; the
// remainders are exact in fp32).  With a ±1 operand every piece's product
// is exact, so three bf16 products accumulate the fp32 product.
__device__ inline void split_bf16x3(const float (&x)[8], bf16x8_t& h, bf16x8_t& md,
                                    bf16x8_t& lo) {
  uint32_t ph[4], pm[4], pl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float a0, a1, b0, b1, c0, c1;
    ph[i] = pk_bf16(x[2 * i], x[2 * i + 1], a0, a1);
    const float r0 = x[2 * i] - a0, r1 = x[2 * i + 1] - a1;
    pm[i] = pk_bf16(r0, r1, b0, b1);
    pl[i] = pk_bf16(r0 - b0, r1 - b1, c0, c1);
  }
  h = __builtin_bit_cast(bf16x8_t, ph);
  md = __builtin_bit_cast(bf16x8_t, pm);
  lo = __builtin_bit_cast(bf16x8_t, pl);
}

// A pointer that is the same on every lane, kept in scalar registers (so
// that a lane offset added to it costs one vector add, and the per-row
// bases are not hoisted into vector registers).
template <typename T>
__device__ inline const T* uniform_ptr(const T* p) {
  const uint64_t x = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return reinterpret_cast<const T*>(((uint64_t)hi << 32) | lo);
}

// A lane's packed sign word, shifted so that the lane's column m of each
// 16-column group g of the word (after dropping the first `skip` bits) sits
// at bit 16g + 15: the top bit of byte 2g + 1.
__device__ inline uint64_t lane_signs(uint64_t w, int skip, int m) {
  return (w >> skip) << (15 - m);
}

// ±1 in bf16 for group g of eight rows' lane_signs words (row u is element
// u): a byte permute moves the group's byte of rows 2i and 2i+1 to bytes 1
// and 3, and the mask-and-xor gives -1 (0xBF80) where the bit is clear and
// +1 (0x3F80) where it is set.
template <int g, typename Row>
__device__ inline bf16x8_t pm1_group(Row row) {
  constexpr uint32_t bi = 2 * (g & 1) + 1;  // byte within the group's 32-bit half
  constexpr uint32_t sel = 0x0Cu | (bi << 8) | (0x0Cu << 16) | ((4u + bi) << 24);
  uint32_t p[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint64_t x0 = row(2 * i), x1 = row(2 * i + 1);
    const uint32_t a = g < 2 ? (uint32_t)x0 : (uint32_t)(x0 >> 32);
    const uint32_t b = g < 2 ? (uint32_t)x1 : (uint32_t)(x1 >> 32);
    p[i] = (__builtin_amdgcn_perm(b, a, sel) & 0x80008000u) ^ 0xBF80BF80u;
  }
  return __builtin_bit_cast(bf16x8_t, p);
}

// pm1_group for a group index known only after unrolling (nt & 3).
template <typename Row>
__device__ inline bf16x8_t pm1_group_at(int g, Row row) {
  switch (g) {
    case 0: return pm1_group<0>(row);
    case 1: return pm1_group<1>(row);
    case 2: return pm1_group<2>(row);
    default: return pm1_group<3>(row);
  }
}

// Partial sums of dW~^T over a chunk of R rows, on the matrix cores:
//   part[c][j][k] = sum_{i in chunk c} s(F_i, k) * β_i dζ_ij.
// One wave per (chunk c, 16 columns j, 16*NT bits k): bf16 MFMA 16x16x32
// with A[j][i] = β_i dζ_ij as three bf16 pieces (its exact split) and
// B[i][k] = s(F_i, k) = ±1 over the 32 rows i = r0 + 32 t + 8q + u (u < 8)
// of step t (lane group q), so every product is exact.  Each run of 64 rows
// (two steps, all of its loads issued together) is summed in fp32 and added
// to fp64 accumulators, runs in row order.  Lane (n, q) ends holding
// outputs (4q + r, n) of each 16x16 tile.
constexpr int kWtRun = 64;  // rows per fp32 run

template <int NT>
__global__ __launch_bounds__(kB) void k_bwd_wtilde_mfma(
    int64_t n, int32_t d_in, int32_t d_out, const uint64_t* __restrict__ F, int64_t ldf,
    const float* __restrict__ beta, const float* __restrict__ dz, int64_t lddz,
    int64_t R, int32_t jtiles, int32_t kgroups, int64_t tasks, double* __restrict__ part) {
  constexpr int NW = NT >= 4 ? NT / 4 : 1;  // packed words a lane reads per row
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (kB / 64) +
                    __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (t >= tasks) return;  // no barrier in this kernel
  const int kg = (int)(t % kgroups);
  const int jt = (int)((t / kgroups) % jtiles);
  const int64_t c = t / ((int64_t)kgroups * jtiles);
  const int m = lane & 15, q = lane >> 4;
  const int j = jt * 16 + m;  // this lane's A column
  const int jc = j < d_out ? j : d_out - 1;
  const int k0 = kg * 16 * NT;
  const int w0 = k0 >> 6;
  const int kw = (d_in + 63) >> 6;
  const int64_t i0 = c * R, i1 = std::min<int64_t>(n, i0 + R);
  const float jm = j < d_out ? 1.f : 0.f;
  const int64_t zoff = (int64_t)(8 * q) * lddz + jc, foff = (int64_t)(8 * q) * ldf;
  int wsel[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) wsel[w] = w0 + w < kw ? w0 + w : kw - 1;
  float4_t acc[NT];
  double acc64[NT][4];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc64[nt][r] = 0.0;
  for (int64_t r0 = i0; r0 < i1; r0 += kWtRun) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = float4_t{0.f, 0.f, 0.f, 0.f};
    // All of the run's loads are issued together, with no branch between
    // them; columns past d_out are zeroed by a 0/1 factor (a select would
    // let the compiler move the loads into a branch and wait on each).
    float a[kWtRun / 4];
    uint64_t wd[kWtRun / 4][NW];
    if (r0 + kWtRun <= i1) {
      // A whole run: row r0 + 32(u/8) + (u%8) (the same on every lane) plus
      // this lane's 8q, so each address is a uniform row base and a fixed
      // lane offset.
#pragma unroll
      for (int u = 0; u < kWtRun / 4; ++u) {
        const int64_t ub = r0 + 32 * (u >> 3) + (u & 7);
        const float* zb = uniform_ptr(dz + ub * lddz);
        const uint64_t* fb = uniform_ptr(F + ub * ldf);
        a[u] = beta[ub + 8 * q] * zb[zoff] * jm;
#pragma unroll
        for (int w = 0; w < NW; ++w) wd[u][w] = fb[foff + wsel[w]];
      }
    } else {
      // The chunk's last run: rows past it read the chunk's last row (an
      // in-range address) and are zeroed by the 0/1 factor.
#pragma unroll
      for (int u = 0; u < kWtRun / 4; ++u) {
        const int64_t row = r0 + 32 * (u >> 3) + 8 * q + (u & 7);
        const int64_t rc = row < i1 ? row : i1 - 1;
        a[u] = beta[rc] * dz[rc * lddz + jc] * (row < i1 ? jm : 0.f);
#pragma unroll
        for (int w = 0; w < NW; ++w) wd[u][w] = F[rc * ldf + wsel[w]];
      }
    }
    __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any MFMA
#pragma unroll
    for (int u = 0; u < kWtRun / 4; ++u)
#pragma unroll
      for (int w = 0; w < NW; ++w) wd[u][w] = lane_signs(wd[u][w], k0 & 63, m);
#pragma unroll
    for (int t = 0; t < kWtRun / 32; ++t) {
      float x8[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x8[u] = a[8 * t + u];
      bf16x8_t ah, am, alo;
      split_bf16x3(x8, ah, am, alo);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const bf16x8_t b =
            pm1_group_at(nt & 3, [&](int u) { return wd[8 * t + u][nt >> 2]; });
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b, acc[nt], 0, 0, 0);
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, b, acc[nt], 0, 0, 0);
        acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, b, acc[nt], 0, 0, 0);
      }
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc64[nt][r] += (double)acc[nt][r];
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int jo = jt * 16 + 4 * q + r;
    if (jo >= d_out) break;
    double* dst = part + ((int64_t)c * d_out + jo) * d_in;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int k = k0 + 16 * nt + m;
      if (k < d_in) dst[k] = acc64[nt][r];
    }
  }
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

// dH~[i][k] = sum_j α_j dζ_ij s(B_j, k) and Eq. (14), on the matrix cores.
// One wave per (16*RT rows, 16*NT columns k): bf16 MFMA 16x16x32 over each
// 32-wide chunk of j with A[i][j] = α_j dζ_ij as three bf16 pieces (its
// exact split) and B[j][k] = s(B_j, k) = ±1, so every product is exact and
// the sum runs in fp32, as a sequential sum would; each ±1 operand is built
// once and used by the RT row tiles and the three pieces.  Lane group q
// takes j = j0 + 8q + s (s < 8), so a lane's eight A values of a row tile
// are two 16-byte loads of its row.  The packed weight words and α sit in
// LDS (rows padded to a multiple of 32 with zeros).
template <int NT, int RT>
__global__ __launch_bounds__(kB) void k_bwd_htilde_mfma(
    int64_t n, int32_t d_in, int32_t d_out, const float* __restrict__ dz, int64_t lddz,
    const uint64_t* __restrict__ B, int64_t ldb, const float* __restrict__ alpha,
    int32_t kgroups, float* __restrict__ dht, int64_t lddht, float* __restrict__ dh,
    int64_t lddh) {
  constexpr int NW = NT >= 4 ? NT / 4 : 1;
  extern __shared__ uint64_t sB[];  // [jpad][kw] words, then α [jpad] (16-byte aligned)
  const int kw = (d_in + 63) >> 6;
  const int jpad = (d_out + 31) & ~31;
  float* sA = reinterpret_cast<float*>(sB + (size_t)jpad * kw);
  for (int idx = threadIdx.x; idx < jpad * kw; idx += kB) {
    const int jj = idx / kw;
    sB[idx] = jj < d_out ? B[(int64_t)jj * ldb + idx % kw] : 0ull;
  }
  for (int jj = threadIdx.x; jj < jpad; jj += kB) sA[jj] = jj < d_out ? alpha[jj] : 0.f;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, q = lane >> 4;
  const int64_t tasks = (n + 16 * RT - 1) / (16 * RT) * kgroups;
  const int64_t nwaves = (int64_t)gridDim.x * (kB / 64);
  for (int64_t t = (int64_t)blockIdx.x * (kB / 64) +
                   __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
       t < tasks; t += nwaves) {
    const int kg = (int)(t % kgroups);
    const int64_t i0 = (t / kgroups) * 16 * RT;
    const int k0 = kg * 16 * NT;
    const int w0 = k0 >> 6;
    float4_t acc[RT][NT];
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[r][nt] = float4_t{0.f, 0.f, 0.f, 0.f};
    // The next chunk's 16-byte loads (clamped to valid addresses: a row past
    // n repeats row n-1, whose outputs are never stored; columns past d_out
    // are zeroed below) are issued before this chunk's MFMAs.
    const float* zr[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const int64_t row = i0 + 16 * r + m;  // this lane's A row in tile r
      zr[r] = dz + (row < n ? row : n - 1) * lddz;
    }
    auto load_chunk = [&](int jn, float4_t (&u0)[RT], float4_t (&u1)[RT]) {
      const int c = jn + 8 * q;
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        u0[r] = *reinterpret_cast<const float4_t*>(zr[r] + (c < d_out ? c : 0));
        u1[r] = *reinterpret_cast<const float4_t*>(zr[r] + (c + 4 < d_out ? c + 4 : 0));
      }
    };
    float4_t n0[RT], n1[RT];
    load_chunk(0, n0, n1);
    for (int j0 = 0; j0 < d_out; j0 += 32) {
      const int jb = j0 + 8 * q;
      float4_t v0[RT], v1[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        v0[r] = n0[r];
        v1[r] = n1[r];
      }
      if (j0 + 32 < d_out) load_chunk(j0 + 32, n0, n1);
      __builtin_amdgcn_sched_barrier(0);
      const float4_t al0 = *reinterpret_cast<const float4_t*>(sA + jb);
      const float4_t al1 = *reinterpret_cast<const float4_t*>(sA + jb + 4);
      bf16x8_t ah[RT], am[RT], alo[RT];
#pragma unroll
      for (int r = 0; r < RT; ++r) {
        float a[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const float v = s < 4 ? v0[r][s] : v1[r][s - 4];
          const float al = s < 4 ? al0[s] : al1[s - 4];
          a[s] = jb + s < d_out ? al * v : 0.f;
        }
        split_bf16x3(a, ah[r], am[r], alo[r]);
      }
      uint64_t wd[8][NW];
#pragma unroll
      for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int w = 0; w < NW; ++w)
          wd[s][w] = lane_signs(w0 + w < kw ? sB[(jb + s) * kw + w0 + w] : 0ull, k0 & 63, m);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const bf16x8_t b = pm1_group_at(nt & 3, [&](int s) { return wd[s][nt >> 2]; });
#pragma unroll
        for (int r = 0; r < RT; ++r) {
          acc[r][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[r], b, acc[r][nt], 0, 0, 0);
          acc[r][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am[r], b, acc[r][nt], 0, 0, 0);
          acc[r][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo[r], b, acc[r][nt], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int64_t ro = i0 + 16 * r + 4 * q + rr;
        if (ro >= n) break;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int k = k0 + 16 * nt + m;
          if (k >= d_in) continue;
          const float v = acc[r][nt][rr];
          if (dht != nullptr) dht[ro * lddht + k] = v;
          if (dh != nullptr) dh[ro * lddh + k] = fabsf(v) < 1.f ? v : 0.f;
        }
      }
  }
}

inline unsigned grid_of(int64_t threads) {
  return (unsigned)std::max<int64_t>(1, (threads + kB - 1) / kB);
}

// Power of two >= v, at most cap.
inline int pow2_at_least(int v, int cap) {
  int p = 1;
  while (p < v && p < cap) p <<= 1;
  return p;
}

// Workspace layout of bigcn_layer_backward, and the tiling of the two
// matrix-core products: dW~ takes 16 x 16*ntw tiles (ntw <= 8), dH~
// 32 x 16*nth tiles (nth <= 8: two row tiles share each ±1 operand), each
// with kgroups tiles across d_in.
struct BwdLayout {
  int64_t kw, ldm, R, chunks, Rdb, chunks_db;
  int ntw, kgw, jtw, nth, kgh;
  size_t off_F, off_beta, off_s, off_ones, off_Gm, off_dz, off_pdb, off_pw, off_wtd,
      off_spmm, bytes;
};

BwdLayout bwd_layout(int64_t n, int64_t nnz, int32_t d_in, int32_t d_out) {
  BwdLayout L;
  L.kw = words(d_in);
  L.ldm = (d_out + 3) / 4 * 4;
  const int ktiles = (d_in + 15) / 16;
  L.ntw = pow2_at_least(ktiles, 8);
  L.kgw = (ktiles + L.ntw - 1) / L.ntw;
  L.jtw = (d_out + 15) / 16;
  L.nth = pow2_at_least(ktiles, 8);
  L.kgh = (ktiles + L.nth - 1) / L.nth;
  // Row chunks of the dW~ partial sums: about 4096 waves of (chunk, 16
  // columns, 16*ntw bits), chunks of at least 256 rows, partial sums within
  // 512 MB.
  const int64_t per_chunk = (int64_t)L.jtw * L.kgw;
  int64_t chunks = std::max<int64_t>(1, 4096 / per_chunk);
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (n + 255) / 256));
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (512ll << 20) / ((int64_t)d_out * d_in * 8)));
  L.R = std::max<int64_t>(1, (n + chunks - 1) / chunks);
  L.chunks = std::max<int64_t>(1, (n + L.R - 1) / L.R);
  L.Rdb = std::max<int64_t>(64, (n + 1023) / 1024);  // at most 1024 row chunks
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

// The bytes of a row-major fp32 matrix argument ([rows][ld], cols used; a
// null pointer or no rows is empty), for overlap tests between arguments.
struct Span {
  const void* p;
  int64_t rows, cols, ld;
  uintptr_t lo() const { return (uintptr_t)p; }
  uintptr_t hi() const { return lo() + (uintptr_t)(((rows - 1) * ld + cols) * 4); }
  bool empty() const { return p == nullptr || rows <= 0 || cols <= 0; }
  bool overlaps(const Span& o) const {
    return !empty() && !o.empty() && lo() < o.hi() && o.lo() < hi();
  }
};

constexpr int kHtildeRowTiles = 2;  // 16-row tiles per wave sharing each ±1 operand

template <int NT>
void launch_htilde(int64_t n, int32_t d_in, int32_t d_out, int32_t kgroups, const float* dz,
                   int64_t lddz, const uint64_t* B, int64_t ldb, const float* alpha,
                   float* dht, int64_t lddht, float* dh, int64_t lddh, hipStream_t s) {
  const int jpad = (d_out + 31) & ~31;
  const size_t lds = (size_t)jpad * words(d_in) * 8 + (size_t)jpad * 4;
  constexpr int RT = kHtildeRowTiles;
  const int64_t tasks = (n + 16 * RT - 1) / (16 * RT) * kgroups;
  const int64_t blocks = std::min<int64_t>((tasks + 3) / 4, 2048);
  hipLaunchKernelGGL((k_bwd_htilde_mfma<NT, RT>), dim3((unsigned)std::max<int64_t>(1, blocks)),
                     dim3(kB), lds, s, n, d_in, d_out, dz, lddz, B, ldb, alpha, kgroups, dht,
                     lddht, dh, lddh);
}

template <int NT>
void launch_wtilde(int64_t n, int32_t d_in, int32_t d_out, const BwdLayout& L,
                   const uint64_t* F, const float* beta, const float* dz, int64_t lddz,
                   double* part, hipStream_t s) {
  const int64_t tasks = L.chunks * L.jtw * L.kgw;
  hipLaunchKernelGGL((k_bwd_wtilde_mfma<NT>), dim3((unsigned)((tasks + 3) / 4)), dim3(kB), 0,
                     s, n, d_in, d_out, F, L.kw, beta, dz, lddz, L.R, L.jtw, L.kgw, tasks,
                     part);
}

}  // namespace

extern "C" {

size_t bigcn_layer_backward_workspace_bytes(int64_t n, int64_t nnz, int32_t d_in,
                                            int32_t d_out) {
  if (n < 0 || nnz < 0 || d_in < 1 || d_out < 1) return 0;
  return bwd_layout(n, nnz, d_in, d_out).bytes;
}

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
  // the source order: both arrays or neither
  if ((slot == nullptr) != (colslot == nullptr)) return BIGCN_EINVAL;
  if (act == BIGCN_ACT_RELU && n > 0 && (out == nullptr || ldo < d_out)) return BIGCN_EINVAL;
  if ((dh != nullptr && lddh < d_in) || (dh_tilde != nullptr && lddht < d_in) ||
      (dwt_tilde != nullptr && lddwt < d_in) || (dzeta != nullptr && lddz < d_out))
    return BIGCN_EINVAL;
  if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(h, 4) || !aligned(wt, 4) ||
      !aligned(wbits, 8) || !aligned(alpha, 4) || !aligned(gout, 4) || !aligned(out, 4) ||
      !aligned(dh, 4) || !aligned(dh_tilde, 4) || !aligned(dwt, 4) ||
      !aligned(dwt_tilde, 4) || !aligned(db, 4) || !aligned(dzeta, 4) ||
      !aligned(slot, 4) || !aligned(colslot, 4))
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
  // G is aggregated in place when no ReLU mask applies, its rows suit the
  // aggregation's 16-byte loads and db (written before) does not overlap it;
  // dζ is written straight to the caller's buffer when its rows suit those
  // loads and it overlaps no other argument (else to the workspace, then
  // copied): the earlier path's results for any arguments.
  const Span sg{gout, n, d_out, ldg}, sz{dzeta, n, d_out, lddz};
  const Span others[] = {{h, n, d_in, ldh},          {gout, n, d_out, ldg},
                         {out, n, d_out, ldo},       {dh, n, d_in, lddh},
                         {dh_tilde, n, d_in, lddht}, {dwt, d_out, d_in, lddw},
                         {dwt_tilde, d_out, d_in, lddwt}, {db, 1, d_out, d_out},
                         {wt, d_out, d_in, ldwt}};
  bool z_alone = true;
  for (const Span& o : others) z_alone = z_alone && !sz.overlaps(o);
  // (in the source order G is always staged: its rows move to their slots)
  const bool g_direct = slot == nullptr && act != BIGCN_ACT_RELU && ldg % 4 == 0 &&
                        aligned(gout, 16) && !sg.overlaps(Span{db, 1, d_out, d_out});
  const bool z_direct =
      dzeta != nullptr && lddz % 4 == 0 && aligned(dzeta, 16) && z_alone;
  float* Gm = g_direct ? nullptr : (float*)(ws + L.off_Gm);
  const float* Gsrc = g_direct ? gout : Gm;
  const int64_t ldsrc = g_direct ? ldg : L.ldm;
  float* dz = z_direct ? dzeta : (float*)(ws + L.off_dz);
  const int64_t ldz = z_direct ? lddz : L.ldm;
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
  {
    int lpr_log2 = 0;
    while ((1 << lpr_log2) * 4 < L.ldm) ++lpr_log2;  // lanes per staged row
    const int64_t rows_per_block = (kB / 64) * (64 >> lpr_log2);
    const bool relu = act == BIGCN_ACT_RELU;
    // (d a multiple of 4 as well: no load reaches past a row's d entries)
    const bool vec = d_out % 4 == 0 && ldg % 4 == 0 && aligned(gout, 16) &&
                     (!relu || (ldo % 4 == 0 && aligned(out, 16)));
    hipLaunchKernelGGL(k_bwd_prep,
                       dim3((unsigned)std::max<int64_t>(1, (n + rows_per_block - 1) /
                                                               rows_per_block)),
                       dim3(kB), 0, s, n, d_out, gout, ldg, out, ldo, relu ? 1 : 0, Gm, L.ldm,
                       rowptr, mean, sc, ones, slot, lpr_log2, vec ? 1 : 0);
  }
  BIGCN_CHECK(hipGetLastError());
  if (db != nullptr) {
    hipLaunchKernelGGL(k_bwd_colsum_part, dim3((unsigned)L.chunks_db), dim3(kB), 0, s, n,
                       d_out, Gsrc, ldsrc, L.Rdb, pdb, slot);
    hipLaunchKernelGGL(k_bwd_colsum_final, dim3(grid_of(d_out)), dim3(kB), 0, s, d_out,
                       L.chunks_db, pdb, db);
    BIGCN_CHECK(hipGetLastError());
  }
  // dζ = Ã^T G: sources scaled by s_i, destinations by D̂^-1/2 (symmetric)
  // or not at all (mean, normalisation mode 2); in the source order the
  // sources are read through the column slots (the same terms in the same
  // order: the results do not change).
  if (n > 0) {
    const bigcn::SpmmPlan plan = bigcn::spmm_plan(n, nnz, d_out);
    BIGCN_CHECK(bigcn::launch_spmm_rows(n, nnz, rowptr, plan, wsp, s));
    BIGCN_CHECK(bigcn::launch_spmm(n, nnz, rowptr, slot != nullptr ? colslot : colidx,
                                   mean ? 2 : 0, sc, Gsrc,
                                   bigcn::IType::F32, d_out, ldsrc, ones, nullptr, 0, dz,
                                   ldz, plan, wsp, s));
    if (dzeta != nullptr && !z_direct)
      BIGCN_CHECK(hipMemcpy2DAsync(dzeta, lddz * 4, dz, L.ldm * 4, (size_t)d_out * 4, n,
                                   hipMemcpyDeviceToDevice, s));
  }
  // dW~^T, then Eq. (15).
  switch (L.ntw) {
    case 1: launch_wtilde<1>(n, d_in, d_out, L, F, beta, dz, ldz, pw, s); break;
    case 2: launch_wtilde<2>(n, d_in, d_out, L, F, beta, dz, ldz, pw, s); break;
    case 4: launch_wtilde<4>(n, d_in, d_out, L, F, beta, dz, ldz, pw, s); break;
    default: launch_wtilde<8>(n, d_in, d_out, L, F, beta, dz, ldz, pw, s); break;
  }
  hipLaunchKernelGGL(k_bwd_wtilde_final, dim3(grid_of((int64_t)d_in * d_out)), dim3(kB), 0,
                     s, d_in, d_out, L.chunks, pw, wtd, dwt_tilde, lddwt);
  hipLaunchKernelGGL(k_bwd_weights, dim3((unsigned)d_out), dim3(kB), 0, s, d_in, wtd, wbits,
                     ldw, alpha, wt, ldwt, dwt, lddw);
  BIGCN_CHECK(hipGetLastError());
  // dH~ and dH (Eq. (14)).
  if (n > 0 && (dh != nullptr || dh_tilde != nullptr)) {
#define BIGCN_HT(NTV)                                                                  \
  launch_htilde<NTV>(n, d_in, d_out, L.kgh, dz, ldz, wbits, ldw, alpha, dh_tilde, lddht, \
                     dh, lddh, s)
    switch (L.nth) {
      case 1: BIGCN_HT(1); break;
      case 2: BIGCN_HT(2); break;
      case 4: BIGCN_HT(4); break;
      default: BIGCN_HT(8); break;
    }
#undef BIGCN_HT
    BIGCN_CHECK(hipGetLastError());
  }
#undef BIGCN_CHECK
  return BIGCN_OK;
}

}  // extern "C"
