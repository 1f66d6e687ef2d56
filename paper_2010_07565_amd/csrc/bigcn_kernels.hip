// gfx950 kernels of the binarized-GCN inference path.
//
//   k_pack        sign binarisation + per-row mean |y| scale (Eqs. (3)-(4),
//                 (7)-(8)); one wave per row, one wave ballot per 64 elements
//                 gives one packed 64-bit word directly.
//   k_bgemm_pop   binary GEMM C = K - 2 popcount(F ^ B) (Eqs. (11)-(12)); the
//                 packed weights sit in LDS, each wave owns a tile of RM rows
//                 whose words arrive through scalar loads, each lane owns CN
//                 output columns; v_xor_b32 + v_bcnt_u32_b32 per 32 bits.
//   k_spmm        aggregation out = act(rowfac * alpha * sum g_j C_j + b)
//                 (Eq. (13) with the rescale of Eq. (11)); the CSR edge range
//                 is cut into equal chunks, one chunk per worker of L lanes,
//                 so hub rows of power-law graphs are shared by many workers;
//                 rows cut by a chunk boundary leave fp32 partial sums that
//                 k_spmm_fix adds in chunk order (no atomics: bitwise
//                 reproducible results).
//
// Wave size is 64 on gfx950 throughout.

#include "bigcn_internal.h"

#include <hip/hip_fp16.h>

#include <type_traits>

namespace bigcn {
namespace {

constexpr int kBlock = 256;  // 4 waves
constexpr int kWavesPerBlock = kBlock / 64;

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef int int4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

// Buffer resource for raw (unformatted) loads: base, stride 0, byte range,
// and the gfx9 default of the fourth descriptor word.  Loads past the range
// return zero.
template <typename T>
__device__ inline __amdgpu_buffer_rsrc_t raw_rsrc(const T* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(p), (short)0, (int)bytes,
                                           0x00020000);
}

constexpr uint32_t kPastEnd = 0x80000000u;  // buffer offset past every range: loads give 0

__device__ inline int wave_index_in_block() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// DPP lane exchange within rows of 16 lanes (quad_perm, row_mirror and
// row_half_mirror controls of gfx9 DPP).
template <int CTRL>
__device__ inline float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                       0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

__device__ inline float wave_sum(float v) {
  // Order-fixed sum, the same in every lane: pairs (xor 1, xor 2), then the
  // mirrored half rows and rows of 16 lanes, then the four rows' sums read
  // out and added as (r0 + r1) + (r2 + r3).
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);  // row_half_mirror
  v += dpp<0x140>(v);  // row_mirror
  const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (a + b) + (c + d);
}

// One level of the row-group sum below: of the partial sums a and b (two
// rows, one register each) a lane keeps one, sends the other to its DPP
// partner and adds what the partner sent, so one register carries both
// rows from here on.
template <int CTRL>
__device__ inline float merge_rows(float a, float b, bool take_b) {
  const float keep = take_b ? b : a;
  const float send = take_b ? a : b;
  return keep + dpp<CTRL>(send);
}

// The wave sums of RW rows (RW in {1, 2, 4, 8}), each formed by exactly the
// additions of wave_sum (same operands, same tree), for about three
// instructions per row instead of thirteen: the first log2(RW) levels of the
// tree merge the rows' registers pairwise.  Lane u of every 16 lanes plays
// place p(u) of its 8-lane half row (the upper half row of 16 mirrored, and
// the upper quad of each half row mirrored), so that the partners of the
// quad_perm, half-mirror and mirror exchanges always carry the same row.
// Lane q < RW returns the sum of row q.
template <int RW>
__device__ inline float rows_sum(const float (&v)[RW], int lane) {
  int u = lane & 15;
  if (u >= 8) u = 15 - u;
  const bool s3 = u >= 4;
  const int c = s3 ? 7 - u : u;
  const bool s1 = (c & 1) != 0, s2 = (c & 2) != 0;
  float t;
  if constexpr (RW == 8) {
    const float p0 = merge_rows<0xB1>(v[0], v[1], s1), p1 = merge_rows<0xB1>(v[2], v[3], s1);
    const float p2 = merge_rows<0xB1>(v[4], v[5], s1), p3 = merge_rows<0xB1>(v[6], v[7], s1);
    const float q0 = merge_rows<0x4E>(p0, p1, s2), q1 = merge_rows<0x4E>(p2, p3, s2);
    t = merge_rows<0x141>(q0, q1, s3);  // lane: row 4 s3 + c
  } else if constexpr (RW == 4) {
    const float p0 = merge_rows<0xB1>(v[0], v[1], s1), p1 = merge_rows<0xB1>(v[2], v[3], s1);
    t = merge_rows<0x4E>(p0, p1, s2);  // lane: row c
    t += dpp<0x141>(t);
  } else if constexpr (RW == 2) {
    t = merge_rows<0xB1>(v[0], v[1], s1);  // lane: row c & 1
    t += dpp<0x4E>(t);
    t += dpp<0x141>(t);
  } else {
    static_assert(RW == 1, "row groups of 1, 2, 4 or 8");
    t = v[0];
    t += dpp<0xB1>(t);
    t += dpp<0x4E>(t);
    t += dpp<0x141>(t);
  }
  t += dpp<0x140>(t);  // rows of 16 lanes
  // the four rows of 16: (r0 + r1) + (r2 + r3)
  t += __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((lane ^ 16) * 4, __builtin_bit_cast(int, t)));
  t += __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute((lane ^ 32) * 4, __builtin_bit_cast(int, t)));
  // a lane carrying row `lane`: place `lane` for rows 0-3, 11 - lane for 4-7
  const int src = lane < RW ? (RW == 8 && lane >= 4 ? 11 - lane : lane) : 0;
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src * 4, __builtin_bit_cast(int, t)));
}

// 8-bit half-codes of one row, NB per lane (lane l: columns l + 64 c), and a
// flagged row's exact products in the same order.
template <int NB>
__device__ inline void store_codes(int8_t* p, uint32_t packed) {
  if constexpr (NB == 4)
    *reinterpret_cast<uint32_t*>(p) = packed;
  else if constexpr (NB == 2)
    *reinterpret_cast<uint16_t*>(p) = (uint16_t)packed;
  else
    *reinterpret_cast<uint8_t*>(p) = (uint8_t)packed;
}

// The low bytes of NB ints as one word (byte c from v[c]), by byte permutes.
template <int NB>
__device__ inline uint32_t pack_low_bytes(const int* v) {
  if constexpr (NB == 4) {
    // v_perm: selector bytes 0-3 take the second operand's bytes, 4-7 the
    // first's, 0x0C gives zero
    const uint32_t lo = __builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x0C0C0400u);
    return __builtin_amdgcn_perm((uint32_t)v[3], (uint32_t)v[2], 0x04000C0Cu) | lo;
  } else if constexpr (NB == 2) {
    return __builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x0C0C0400u);
  } else {
    return (uint32_t)v[0] & 0xFFu;
  }
}

// store_codes for a row address the whole wave shares: a buffer resource
// built on the scalar unit and a lane offset, no per-lane address math.
template <int NB>
__device__ inline void store_codes_row(int8_t* row, int lane, uint32_t packed) {
  const __amdgpu_buffer_rsrc_t rs = raw_rsrc(row, 64u * NB);
  if constexpr (NB == 4)
    __builtin_amdgcn_raw_buffer_store_b32(packed, rs, lane * 4, 0, 0);
  else if constexpr (NB == 2)
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)packed, rs, lane * 2, 0, 0);
  else
    __builtin_amdgcn_raw_buffer_store_b8((uint8_t)packed, rs, lane, 0, 0);
}

template <int NB>
__device__ inline void store_exact(_Float16* p, const int* v) {
  if constexpr (NB == 4) {
    half4_t h;
#pragma unroll
    for (int c = 0; c < 4; ++c) h[c] = (_Float16)v[c];
    *reinterpret_cast<half4_t*>(p) = h;
  } else if constexpr (NB == 2) {
    half2_t h;
    h[0] = (_Float16)v[0];
    h[1] = (_Float16)v[1];
    *reinterpret_cast<half2_t*>(p) = h;
  } else {
    *p = (_Float16)v[0];
  }
}

// ---------------------------------------------------------------- pack ----

template <bool STD>
__global__ __launch_bounds__(kBlock) void k_pack(
    const float* __restrict__ x, int64_t rows, int32_t cols, int64_t ldx,
    const float* __restrict__ mu, const float* __restrict__ rstd,
    const int64_t* __restrict__ rowptr, int sym, uint64_t* __restrict__ bits,
    int64_t ldw, float* __restrict__ scale, const int32_t* __restrict__ slot) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = (int64_t)gridDim.x * kWavesPerBlock;
  const int kw = (cols + 63) >> 6;
  for (int64_t r = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
       r < rows; r += nwaves) {
    const float* xr = x + r * ldx;
    const int64_t dst = slot != nullptr ? (int64_t)slot[r] : r;
    uint64_t* br = bits + dst * ldw;
    float l1 = 0.f;
    for (int64_t wb = 0; wb < ldw; wb += 64) {
      // Lane q keeps word wb + q of this batch of 64 words.
      uint64_t mine = 0;
      const int wend = (int)(wb + 64 < kw ? wb + 64 : kw);
      int w = (int)wb;
      for (; w + 4 <= wend; w += 4) {
        float v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int k = (w + u) * 64 + lane;
          v[u] = k < cols ? xr[k] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int k = (w + u) * 64 + lane;
          const bool ok = k < cols;
          float y = v[u];
          if (STD && ok) {
            const float t = y - mu[k];  // two separate fp32 roundings
            y = t * rstd[k];
          }
          const uint64_t b = __builtin_amdgcn_ballot_w64(ok && y >= 0.f);
          l1 += ok ? fabsf(y) : 0.f;
          if (lane == (int)(w + u - wb)) mine = b;
        }
      }
      for (; w < wend; ++w) {
        const int k = w * 64 + lane;
        const bool ok = k < cols;
        float y = ok ? xr[k] : 0.f;
        if (STD && ok) {
          const float t = y - mu[k];
          y = t * rstd[k];
        }
        const uint64_t b = __builtin_amdgcn_ballot_w64(ok && y >= 0.f);
        l1 += ok ? fabsf(y) : 0.f;
        if (lane == (int)(w - wb)) mine = b;
      }
      if (wb + lane < ldw) br[wb + lane] = mine;  // pad words stay zero
    }
    l1 = wave_sum(l1);
    if (lane == 0) {
      float s = l1 / (float)cols;
      if (rowptr != nullptr && sym) {
        const int64_t dg = rowptr[r + 1] - rowptr[r];
        s = s * (dg > 0 ? 1.0f / sqrtf((float)dg) : 0.f);
      }
      scale[dst] = s;
    }
  }
}

// Row stride limit of k_pack_rows, whose RW-row groups are addressed with
// 32-bit buffer offsets.
constexpr int64_t kPackRowsMaxLd = (int64_t)1 << 24;

// Same computation with RW rows per wave in flight: all RW*kw loads of a
// row group are issued before the first ballot, and the RW row sums are
// reduced together.  kw <= KWT <= 32 and RW * ldw <= 64: lane RW q + w
// collects word w of row q, so the group's words (rows r0.. contiguous at
// stride ldw) and scales leave in one store each.
// With NBQ > 0 the binary GEMM of a layer of N <= 64 NBQ outputs follows in
// place (lane l: outputs l + 64 c for c < NBQ, their weight words in
// registers, KWT NBQ <= 16; the row's words are the ballots): the 8-bit
// half-codes, exact rows and flags of k_bgemm_pop_q8 (NBQ bytes per lane, the
// interleaved row layout) are written instead of the bits.
// With slot != nullptr row r's results go to row slot[r] of bits / scale /
// codes (the source order of the aggregation); else to row r.

template <bool STD, int RW, int KWT, int NBQ>
__global__ __launch_bounds__(kBlock) void k_pack_rows(
    const float* __restrict__ x, int64_t rows, int32_t cols, int64_t ldx,
    const float* __restrict__ mu, const float* __restrict__ rstd,
    const int64_t* __restrict__ rowptr, int sym, uint64_t* __restrict__ bits,
    int64_t ldw, float* __restrict__ scale, const uint64_t* __restrict__ B, int32_t N,
    int64_t ldb, int8_t* __restrict__ C8, int64_t ldc8, _Float16* __restrict__ C16,
    int64_t ldc16, const int32_t* __restrict__ slot) {
  // Column statistics: in registers (lane l keeps columns 64 w + l) up to
  // 16 words, so the first row loads need not wait for a block barrier;
  // in LDS (mu[0..cols), rstd[cols..2 cols)) for wider rows.
  extern __shared__ float s_norm[];
  constexpr bool FQ = NBQ > 0;
  constexpr int NQ = FQ ? NBQ : 1;
  constexpr bool kNLds = STD && KWT > 16;
  const int lane = threadIdx.x & 63;
  const int kw = (cols + 63) >> 6;
  float mr[STD && !kNLds ? KWT : 1], rr[STD && !kNLds ? KWT : 1];
  if constexpr (STD && !kNLds) {
    // columns past cols fall outside the ranges and read as zero
    const __amdgpu_buffer_rsrc_t rsm = raw_rsrc(mu, (uint32_t)cols * 4u);
    const __amdgpu_buffer_rsrc_t rsr = raw_rsrc(rstd, (uint32_t)cols * 4u);
#pragma unroll
    for (int w = 0; w < KWT; ++w) {
      const uint32_t off = w < kw ? (uint32_t)(w * 64 + lane) * 4u : kPastEnd;
      mr[w] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsm, (int)off, 0, 0));
      rr[w] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsr, (int)off, 0, 0));
    }
  }
  if (kNLds) {
    for (int i = threadIdx.x; i < cols; i += kBlock) {
      s_norm[i] = mu[i];
      s_norm[cols + i] = rstd[i];
    }
    __syncthreads();
  }
  // With the statistics in registers, lanes past cols load zero (their
  // statistics are zero too), so their |y| adds zero without a mask.
  constexpr bool kZeroPad = !kNLds;
  // 8-bit codes (cols - cols % 2) / 2 - popcount leave [-128, 127] only
  // for rows of more than 255 inputs.
  const int half = (cols - (cols & 1)) >> 1;
  const bool may_big = cols > 255;
  const int64_t step = (int64_t)gridDim.x * kWavesPerBlock * RW;
  static_assert(!FQ || KWT * NBQ <= 16, "fused GEMM keeps its weight words in registers");
  uint64_t wr[NQ][FQ ? KWT : 1];  // FQ: the words of lane l's columns l + 64 c
  if constexpr (FQ) {
    const __amdgpu_buffer_rsrc_t rsb = raw_rsrc(B, (uint32_t)(N * ldb * 8));
#pragma unroll
    for (int c = 0; c < NQ; ++c) {
      const int col = lane + 64 * c;
#pragma unroll
      for (int w = 0; w < KWT; ++w) {
        const uint32_t off =
            (col < N && w < kw) ? (uint32_t)(col * ldb + w) * 8u : kPastEnd;
        wr[c][w] = __builtin_bit_cast(
            uint64_t, __builtin_amdgcn_raw_buffer_load_b64(rsb, (int)off, 0, 0));
      }
    }
  }
  // Lane offset of word w within a row (the row's own offset q ldx is the
  // scalar offset of its loads); lanes past cols read past the range: zero.
  uint32_t voff[KWT];
#pragma unroll
  for (int w = 0; w < KWT; ++w)
    voff[w] = !kZeroPad || w * 64 + lane < cols ? (uint32_t)(w * 64 + lane) * 4u : kPastEnd;
  for (int64_t r0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block()) * RW;
       r0 < rows; r0 += step) {
    // The group's nq rows as one raw buffer ending with the last row's
    // element cols - 1 (element (q, k) at byte 4 (q ldx + k)); without
    // kZeroPad elements past cols in a row are loaded but masked below.
    // Every load is issued before any result is used.
    const int nq = (int)(rows - r0 < RW ? rows - r0 : RW);
    const __amdgpu_buffer_rsrc_t rsx =
        raw_rsrc(x + r0 * ldx, (uint32_t)(((nq - 1) * ldx + cols) * 4));
    // lane q < nq: the output row of row r0 + q (the fused GEMM stores each
    // row's codes as soon as they are formed, so it is loaded first)
    int32_t dq = 0;
    if (FQ && slot != nullptr) dq = slot[r0 + (lane < nq ? lane : 0)];
    // Rows past the matrix (q >= nq, last group only) load row nq - 1
    // again, so no scalar offset leaves the range; nothing of theirs is
    // stored.
    float v[RW][KWT];
#pragma unroll
    for (int q = 0; q < RW; ++q) {
      const int qo = (q < nq ? q : nq - 1) * (int)ldx * 4;
#pragma unroll
      for (int w = 0; w < KWT; ++w)
        v[q][w] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(rsx, (int)voff[w], qo, 0));
    }
    // lane q < nq: the degree of row r0 + q (for the normalisation factor),
    // loaded after the rows so that waiting for it does not hold them back
    int64_t dg = 0;
    if (rowptr != nullptr && sym) {
      const int64_t rq = r0 + (lane < nq ? lane : 0);
      dg = rowptr[rq + 1] - rowptr[rq];
    }
    if (!FQ && slot != nullptr) dq = slot[r0 + (lane < nq ? lane : 0)];
    float l1[RW];
    uint64_t mine = 0;  // lane ldw q + w: word w of row q (pad words stay zero)
    bool myflag = false;  // FQ, lane q < nq: row r0 + q has exact products
#pragma unroll
    for (int q = 0; q < RW; ++q) {
      l1[q] = 0.f;
      int pc[NQ];  // FQ: popcount of row XOR the weights of column lane + 64 c
#pragma unroll
      for (int c = 0; c < NQ; ++c) pc[c] = 0;
#pragma unroll
      for (int w = 0; w < KWT; ++w) {
        if (w >= kw) continue;  // wave-uniform (every later word too)
        // Lanes past cols hold zero (kZeroPad) or junk (the next row or
        // zero): the last word's lane mask drops their bits and its sum
        // skips them.
        const bool full = (w + 1) * 64 <= cols;  // wave-uniform
        float y = v[q][w];
        if constexpr (STD) {
          // two separate fp32 roundings
          const int k = w * 64 + lane;
          const int kk = kNLds && k >= cols ? 0 : k;
          const float t = y - (kNLds ? s_norm[kk] : mr[w]);
          y = t * (kNLds ? s_norm[cols + kk] : rr[w]);
        }
        uint64_t b = __builtin_amdgcn_fcmpf(y, 0.f, 3 /* ordered >= */);
        if (!full) b &= (1ull << (cols & 63)) - 1;
        if (kZeroPad || full)
          l1[q] += fabsf(y);
        else
          l1[q] += lane < (cols & 63) ? fabsf(y) : 0.f;
        if (!FQ && lane == q * ldw + w) mine = b;
        if constexpr (FQ) {
#pragma unroll
          for (int c = 0; c < NQ; ++c) {
            const uint64_t z = b ^ wr[c][w];
            pc[c] = __builtin_popcount((uint32_t)(z >> 32)) +
                    (__builtin_popcount((uint32_t)z) + pc[c]);
          }
        }
      }
      if constexpr (FQ) {
        if (q < nq) {  // wave-uniform
          const int64_t dr =
              slot != nullptr ? (int64_t)__builtin_amdgcn_readlane(dq, q) : r0 + q;
          int code[NQ];
#pragma unroll
          for (int c = 0; c < NQ; ++c)
            code[c] = half - pc[c];  // (dot - cols % 2) / 2, dot = cols - 2 popcount
          store_codes_row<NQ>(C8 + dr * ldc8, lane, pack_low_bytes<NQ>(code));
          if (may_big) {
            bool big = false;
#pragma unroll
            for (int c = 0; c < NQ; ++c)
              big |= lane + 64 * c < N && (code[c] < -128 || code[c] > 127);
            const bool flag = __builtin_amdgcn_ballot_w64(big) != 0;
            if (flag) {
              int dot[NQ];
#pragma unroll
              for (int c = 0; c < NQ; ++c) dot[c] = cols - 2 * pc[c];
              store_exact<NQ>(C16 + dr * ldc16 + NQ * lane, dot);
            }
            if (lane == q) myflag = flag;
          }
        }
      }
    }
    // lane q < nq: row r0 + q's sum
    const float myl1 = rows_sum<RW>(l1, lane);
    if constexpr (!FQ) {
      if (slot == nullptr) {
        if (lane < nq * ldw) bits[r0 * ldw + lane] = mine;
      } else {  // word lane % ldw of row lane / ldw, at that row's slot
        const int q = lane / (int)ldw;
        const int dr = __builtin_amdgcn_ds_bpermute((q < RW ? q : 0) * 4, dq);  // all lanes
        if (lane < nq * ldw) bits[(int64_t)dr * ldw + (lane - q * (int)ldw)] = mine;
      }
    }
    if (lane < nq) {
      float sc = myl1 / (float)cols;
      if (rowptr != nullptr && sym) sc = sc * (dg > 0 ? 1.0f / sqrtf((float)dg) : 0.f);
      scale[slot != nullptr ? (int64_t)dq : r0 + lane] = myflag ? -fabsf(sc) : sc;
    }
  }
}

// ------------------------------------------------------ bgemm (popcount) ----

template <typename T>
struct Vec4;
template <>
struct Vec4<_Float16> { typedef half4_t type; };
template <>
struct Vec4<int16_t> { typedef short4_t type; };
template <>
struct Vec4<int32_t> { typedef int4_t type; };
template <>
struct Vec4<float> { typedef float4_t type; };

template <typename T>
__device__ inline T from_int(int v) { return (T)v; }

// Stores CN consecutive results of one row.
template <typename T, int CN>
__device__ inline void store_row(T* __restrict__ dst, const int* v, int ncols,
                                 bool vec) {
  if (CN == 4 && vec && ncols >= 4) {
    typename Vec4<T>::type p;
    p[0] = from_int<T>(v[0]);
    p[1] = from_int<T>(v[1]);
    p[2] = from_int<T>(v[2]);
    p[3] = from_int<T>(v[3]);
    *reinterpret_cast<typename Vec4<T>::type*>(dst) = p;
    return;
  }
#pragma unroll
  for (int c = 0; c < CN; ++c)
    if (c < ncols) dst[c] = from_int<T>(v[c]);
}

// Stages packed weight rows into LDS as [kw][CN][64]: entry (w*CN + c)*64 + l
// holds word w of the column lane l owns in slot c, so that for a fixed
// (w, c) the 64 lanes read 64 consecutive words.  Lane l owns columns
// j0 + CN*l + c (consecutive) or, with IL, l + 64*c (lane-interleaved).
template <int CN, bool IL = false>
__device__ inline void stage_weights(uint64_t* sB, const uint64_t* __restrict__ B,
                                     int32_t N, int64_t ldb, int kw, int j0) {
  for (int idx = threadIdx.x; idx < kw * CN * 64; idx += kBlock) {
    const int l = idx & 63;
    const int c = (idx >> 6) % CN;
    const int w = idx / (64 * CN);
    const int j = IL ? l + 64 * c : j0 + l * CN + c;
    sB[idx] = j < N ? B[(int64_t)j * ldb + w] : 0ull;
  }
  __syncthreads();
}

// Disagreement counts popcount(F_i ^ B_j) of rows i0 .. i0+RM-1 against this
// lane's CN columns.  The row words are wave-uniform (scalar loads).
template <int CN, int RM>
__device__ inline void tile_popcounts(const uint64_t* __restrict__ F, int64_t M,
                                      int64_t ldf, const uint64_t* sB, int kw,
                                      int64_t i0, int lane, uint32_t (&acc)[RM][CN]) {
#pragma unroll
  for (int r = 0; r < RM; ++r)
#pragma unroll
    for (int c = 0; c < CN; ++c) acc[r][c] = 0;
  for (int w = 0; w < kw; ++w) {
    uint64_t fw[RM];
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      const int64_t i = i0 + r < M ? i0 + r : M - 1;
      fw[r] = F[i * ldf + w];
    }
    uint64_t bw[CN];
#pragma unroll
    for (int c = 0; c < CN; ++c) bw[c] = sB[(w * CN + c) * 64 + lane];
#pragma unroll
    for (int r = 0; r < RM; ++r)
#pragma unroll
      for (int c = 0; c < CN; ++c) {
        const uint64_t z = fw[r] ^ bw[c];
        acc[r][c] += __builtin_popcount((uint32_t)z);
        acc[r][c] += __builtin_popcount((uint32_t)(z >> 32));
      }
  }
}

template <int CN, int RM, typename T>
__global__ __launch_bounds__(kBlock) void k_bgemm_pop(
    const uint64_t* __restrict__ F, int64_t M, int64_t ldf,
    const uint64_t* __restrict__ B, int32_t N, int64_t ldb, int32_t K,
    T* __restrict__ C, int64_t ldc, int vec) {
  extern __shared__ uint64_t sB[];
  const int lane = threadIdx.x & 63;
  const int kw = (K + 63) >> 6;
  const int j0 = blockIdx.y * 64 * CN;
  stage_weights<CN>(sB, B, N, ldb, kw, j0);
  const int64_t tiles = (M + RM - 1) / RM;
  const int64_t nwaves = (int64_t)gridDim.x * kWavesPerBlock;
  const int jl = j0 + lane * CN;  // first column of this lane
  const int ncols = N - jl;       // valid columns from jl (may be <= 0)
  for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
       t < tiles; t += nwaves) {
    const int64_t i0 = t * RM;
    uint32_t acc[RM][CN];
    tile_popcounts<CN, RM>(F, M, ldf, sB, kw, i0, lane, acc);
    if (ncols > 0) {
#pragma unroll
      for (int r = 0; r < RM; ++r) {
        if (i0 + r >= M) break;
        int v[CN];
#pragma unroll
        for (int c = 0; c < CN; ++c) v[c] = K - 2 * (int)acc[r][c];
        store_row<T, CN>(C + (i0 + r) * ldc + jl, v, ncols, vec != 0);
      }
    }
  }
}

// The same product stored as exact 8-bit half-codes for the forward pass:
//   code = (dot - p) / 2,  p = K mod 2   (dot = K - 2 popcount is = p mod 2),
// which holds every |dot| <= 255.  A row holds 64*NB bytes (NB = 1, 2, 4 for
// up to 64, 128, 256 outputs) in lane-interleaved order: column k sits at
// byte NB*(k % 64) + k / 64, so that lane l finds its columns l + 64c
// (c < NB) in one NB-byte word.  A row with a larger |dot| anywhere is
// written in full, exactly, to C16 (IEEE half, the same interleaved order,
// 64*NB halves per row) and flagged by setting the sign bit of its scale
// g[i] (g >= 0 otherwise).  One wave covers all N columns, so the flag is
// decided per row with a ballot.

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float2_t __attribute__((ext_vector_type(2)));

template <int RM, int NB>
__global__ __launch_bounds__(kBlock) void k_bgemm_pop_q8(
    const uint64_t* __restrict__ F, int64_t M, int64_t ldf,
    const uint64_t* __restrict__ B, int32_t N, int64_t ldb, int32_t K,
    int8_t* __restrict__ C8, int64_t ldc8, _Float16* __restrict__ C16,
    int64_t ldc16, float* __restrict__ g) {
  extern __shared__ uint64_t sB[];
  const int lane = threadIdx.x & 63;
  const int kw = (K + 63) >> 6;
  stage_weights<NB, true>(sB, B, N, ldb, kw, 0);
  const int64_t tiles = (M + RM - 1) / RM;
  const int64_t nwaves = (int64_t)gridDim.x * kWavesPerBlock;
  const int par = K & 1;
  for (int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
       t < tiles; t += nwaves) {
    const int64_t i0 = t * RM;
    uint32_t acc[RM][NB];
    tile_popcounts<NB, RM>(F, M, ldf, sB, kw, i0, lane, acc);
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (i0 + r >= M) break;  // wave-uniform
      const int64_t i = i0 + r;
      int v[NB];
      bool big = false;
      uint32_t packed = 0;
#pragma unroll
      for (int c = 0; c < NB; ++c) {
        v[c] = K - 2 * (int)acc[r][c];
        const int code = (v[c] - par) >> 1;
        big |= (lane + 64 * c < N) && (code < -128 || code > 127);
        packed |= (uint32_t)(uint8_t)(int8_t)code << (8 * c);
      }
      store_codes<NB>(C8 + i * ldc8 + NB * lane, packed);
      if (__builtin_amdgcn_ballot_w64(big) != 0) {
        store_exact<NB>(C16 + i * ldc16 + NB * lane, v);
        if (lane == 0) g[i] = -fabsf(g[i]);
      }
    }
  }
}

// ------------------------------------------------------------ bgemm (MFMA) --
//
// The same product on the matrix cores.  With a, b in {0,1} the sign bits
// (pad bits are 0) and s = 2a - 1, for k < K:
//     sum s_a s_b = 4 sum a b - 2 sum a - 2 sum b + K,
// so the signs are expanded to {0,1} bytes and v_mfma_i32_16x16x64_i8 forms
// sum a b exactly over one 64-bit word per instruction.  Operand layout
// (gfx950): lane l of A holds row l % 16, bytes 16*(l/16) .. +15 of the word;
// lane l of B holds column l % 16 with the same bytes; lane L, register R of
// the result holds row 4*(L/16) + R, column L % 16.
// Work split: a block owns one group of NT column tiles (NT*16 <= 128
// columns) and walks row tiles of 4 waves x 32 rows; each wave's two 16-row
// tiles share every weight operand.  The block stages kc words of its
// columns' weights, already expanded, in LDS in B-operand order
// ([word][tile][lane] x 16 bytes: each operand load is one conflict-free
// 16-byte read).  When kc covers all of K the staged weights are kept for
// every row tile of the block (grid is a multiple of the group count, so a
// block's group never changes).  The next feature word is loaded before the
// current word's MFMAs are issued.

typedef int int4v_t __attribute__((ext_vector_type(4)));

// 16 sign bits -> 16 bytes of {0,1} (bit q of each nibble to byte q).
__device__ inline int4v_t expand16(uint32_t bits) {
  int4v_t r;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint32_t nib = (bits >> (4 * q)) & 0xFu;
    r[q] = (int)((nib * 0x00204081u) & 0x01010101u);
  }
  return r;
}

constexpr int kMfmaLdsBytes = 48 * 1024;  // staged weights per block

template <int NT, typename T>
__global__ __launch_bounds__(kBlock) void k_bgemm_mfma(
    const uint64_t* __restrict__ F, int64_t M, int64_t ldf,
    const uint64_t* __restrict__ B, int32_t N, int64_t ldb, int32_t K,
    T* __restrict__ C, int64_t ldc, int32_t groups, int32_t kc_max) {
  extern __shared__ int4v_t sW[];                       // [kc][NT][64]
  __shared__ int sPb[NT * 16];                          // sum b per column
  const int lane = threadIdx.x & 63;
  const int wv = wave_index_in_block();
  const int kw = (K + 63) >> 6;
  const int m = lane & 15, grp = lane >> 4;
  const int cg = blockIdx.x % groups;
  const int c0 = cg * NT * 16;
  for (int j = threadIdx.x; j < NT * 16; j += kBlock) {
    int pc = 0;
    if (c0 + j < N)
      for (int w = 0; w < kw; ++w) pc += __builtin_popcountll(B[(int64_t)(c0 + j) * ldb + w]);
    sPb[j] = pc;
  }
  const bool resident = kc_max >= kw;
  bool staged = false;
  const int64_t rows_per_block = kWavesPerBlock * 32;
  const int64_t row_step = (int64_t)(gridDim.x / groups) * rows_per_block;
  for (int64_t base = (int64_t)(blockIdx.x / groups) * rows_per_block; base < M;
       base += row_step) {
    const int64_t r0 = base + wv * 32;  // this wave: rows r0 .. r0+31
    const int64_t rowA = r0 + m, rowB = r0 + 16 + m;
    const uint64_t* fa = F + (rowA < M ? rowA : 0) * ldf;
    const uint64_t* fb = F + (rowB < M ? rowB : 0) * ldf;
    int4v_t acc[2][NT];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int jt = 0; jt < NT; ++jt) acc[t][jt] = int4v_t{0, 0, 0, 0};
    int pa0 = 0, pa1 = 0;
    for (int w0 = 0; w0 < kw; w0 += kc_max) {
      const int kc = kw - w0 < kc_max ? kw - w0 : kc_max;
      if (!(resident && staged)) {
        __syncthreads();  // previous chunk fully consumed
        for (int idx = threadIdx.x; idx < kc * NT * 64; idx += kBlock) {
          const int l = idx & 63;
          const int jt = (idx >> 6) % NT;
          const int w = idx / (64 * NT);
          const int col = c0 + jt * 16 + (l & 15);
          const uint64_t word = col < N ? B[(int64_t)col * ldb + w0 + w] : 0ull;
          sW[(w * NT + jt) * 64 + l] =
              expand16((uint32_t)(word >> (16 * (l >> 4))) & 0xFFFFu);
        }
        __syncthreads();
        staged = true;
      }
      uint64_t na = rowA < M ? fa[w0] : 0ull;
      uint64_t nb = rowB < M ? fb[w0] : 0ull;
      for (int w = 0; w < kc; ++w) {
        const uint64_t f0 = na, f1 = nb;
        if (w + 1 < kc) {
          na = rowA < M ? fa[w0 + w + 1] : 0ull;
          nb = rowB < M ? fb[w0 + w + 1] : 0ull;
        }
        pa0 += __builtin_popcountll(f0);
        pa1 += __builtin_popcountll(f1);
        const int4v_t a0 = expand16((uint32_t)(f0 >> (16 * grp)) & 0xFFFFu);
        const int4v_t a1 = expand16((uint32_t)(f1 >> (16 * grp)) & 0xFFFFu);
#pragma unroll
        for (int jt = 0; jt < NT; ++jt) {
          const int4v_t bop = sW[(w * NT + jt) * 64 + lane];
          acc[0][jt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0, bop, acc[0][jt], 0, 0, 0);
          acc[1][jt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1, bop, acc[1][jt], 0, 0, 0);
        }
      }
    }
    // Lanes m, m+16, m+32, m+48 all hold row m's full popcount.
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int pa = t == 0 ? pa0 : pa1;
#pragma unroll
      for (int R = 0; R < 4; ++R) {
        const int mr = 4 * grp + R;                     // output row in the tile
        const int pa_r = __shfl(pa, mr, 64);
        const int64_t row = r0 + t * 16 + mr;
#pragma unroll
        for (int jt = 0; jt < NT; ++jt) {
          const int col = c0 + jt * 16 + m;
          if (row < M && col < N) {
            const int dot = K - 2 * (pa_r + sPb[jt * 16 + m]) + 4 * acc[t][jt][R];
            C[row * ldc + col] = (T)dot;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ spmm ----

template <typename T>
__device__ inline typename Vec4<T>::type load4(const T* p) {
  return *reinterpret_cast<const typename Vec4<T>::type*>(p);
}

// acc[c] += g * v[c], one fused multiply-add per element; for half inputs
// this is a single v_fma_mix_f32 (the conversion is exact).
template <typename V>
__device__ inline void fma4(float4_t& acc, float g, const V& v) {
  acc[0] = fmaf((float)v[0], g, acc[0]);
  acc[1] = fmaf((float)v[1], g, acc[1]);
  acc[2] = fmaf((float)v[2], g, acc[2]);
  acc[3] = fmaf((float)v[3], g, acc[3]);
}

struct Epi {
  float alpha[4];
  float bias[4];
  int ncols;  // valid columns of this lane (0..4)
  int relu;
  bool vec;   // 16-byte output stores allowed
};

__device__ inline float act(float v, int relu) { return relu ? fmaxf(v, 0.f) : v; }

__device__ inline void store_out(float* __restrict__ o, const Epi& ep,
                                 const float4_t v) {
  if (ep.vec && ep.ncols == 4) {
    *reinterpret_cast<float4_t*>(o) = v;
    return;
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (c < ep.ncols) o[c] = v[c];
}

__device__ inline void write_row(float* __restrict__ out, int64_t ldo, int64_t r,
                                 int c0, const Epi& ep, const float4_t acc,
                                 float rowfac) {
  float4_t v;
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = act(fmaf(acc[c], rowfac * ep.alpha[c], ep.bias[c]), ep.relu);
  store_out(out + r * ldo + c0, ep, v);
}

__device__ inline void write_empty(float* __restrict__ out, int64_t ldo,
                                   int64_t r, int c0, const Epi& ep) {
  float4_t v;
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = act(ep.bias[c], ep.relu);
  store_out(out + r * ldo + c0, ep, v);
}

// Destination-side factor of Ã for a row with deg entries: D̂^-1/2 (mean 0,
// symmetric), D̂^-1 (mean 1), or none (mean 2: the transpose of the mean
// normalisation, whose factor sits on the source side).
__device__ inline float row_factor_deg(int64_t deg, int mean) {
  const float dg = (float)deg;
  return mean == 2 ? 1.0f : mean ? 1.0f / dg : 1.0f / sqrtf(dg);
}

__device__ inline float row_factor(const int64_t* __restrict__ rowptr, int64_t r,
                                   int mean) {
  return row_factor_deg(rowptr[r + 1] - rowptr[r], mean);
}

// Worker w owns edges [w*chunk, min((w+1)*chunk, nnz)).  It aggregates every
// row that starts inside its range and ends inside it; the row that reaches
// past the range end leaves a "tail" partial (plus tail_row[w]); a row that
// began before the range leaves a "head" partial.  Empty rows are written as
// act(bias) by the worker whose range holds their position.
//
// Latency hiding: column indices are fetched one group of U edges ahead of
// the group whose g / C rows are being gathered, and the ends of the next
// four rows are kept in a small queue that is refilled as rows finish.  With
// L == 64 the worker is the whole wave, so edge and row bookkeeping is
// wave-uniform and lives in scalar registers.
template <int L, typename T, int U>
__global__ __launch_bounds__(kBlock) void k_spmm(
    int64_t n, int64_t nnz, const int64_t* __restrict__ rowptr,
    const int32_t* __restrict__ colidx, int mean, const float* __restrict__ g,
    const T* __restrict__ C, int32_t d, int64_t ldc,
    const float* __restrict__ alpha, const float* __restrict__ bias, int relu,
    float* __restrict__ out, int64_t ldo, int vec_out, int64_t chunk,
    int64_t workers, int32_t dpad, const int32_t* __restrict__ row_of,
    int32_t* __restrict__ tail_row, float* __restrict__ head,
    float* __restrict__ tail) {
  typedef typename Vec4<T>::type V;
  constexpr int P = 64 / L;
  const int lane = threadIdx.x & 63;
  const int slot = L == 64 ? 0 : lane / L;
  if (slot >= P) return;  // idle lanes when L does not divide 64
  const int sub = lane - slot * L;
  const int64_t w =
      ((int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block()) * P + slot;
  if (w >= workers) return;
  const int c0 = blockIdx.y * (L * 4) + sub * 4;
  Epi ep;
  ep.ncols = d - c0 < 0 ? 0 : (d - c0 > 4 ? 4 : d - c0);
  ep.relu = relu;
  ep.vec = vec_out != 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    ep.alpha[c] = c < ep.ncols ? alpha[c0 + c] : 0.f;
    ep.bias[c] = (c < ep.ncols && bias != nullptr) ? bias[c0 + c] : 0.f;
  }
  const bool load_cols = ep.ncols > 0;
  const int64_t kEnd = INT64_MAX;

  const int64_t s = w * chunk;
  const int64_t t = s + chunk < nnz ? s + chunk : nnz;
  int32_t jn[U];  // first group's column indices: independent of the row lookup
#pragma unroll
  for (int u = 0; u < U; ++u) jn[u] = s + u < t ? colidx[s + u] : -1;
  int64_t r = row_of[w];
  int64_t cur_beg = rowptr[r];
  int64_t q1 = r + 2 <= n ? rowptr[r + 2] : kEnd;
  int64_t q2 = r + 3 <= n ? rowptr[r + 3] : kEnd;
  int64_t q3 = r + 4 <= n ? rowptr[r + 4] : kEnd;
  int64_t cur_end = rowptr[r + 1];
  bool before = cur_beg < s;
  if (!before) {
    for (int64_t q = r - 1; q >= 0 && rowptr[q] == s; --q)
      write_empty(out, ldo, q, c0, ep);
  }
  float4_t a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};

  for (int64_t e = s; e < t; e += U) {
    int32_t jj[U];
    float gg[U];
    V vv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) jj[u] = jn[u];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      gg[u] = jj[u] >= 0 ? g[jj[u]] : 0.f;
      if (jj[u] >= 0 && load_cols)
        vv[u] = load4<T>(C + (int64_t)jj[u] * ldc + c0);
      else
        vv[u] = V{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) jn[u] = e + U + u < t ? colidx[e + U + u] : -1;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t eu = e + u;
      if (eu >= t) break;
      if (eu == cur_end) {
        // Row r is finished inside this range.
        const float4_t sum = a0 + a1;
        if (before) {
          if (load_cols) *reinterpret_cast<float4_t*>(head + w * dpad + c0) = sum;
        } else {
          write_row(out, ldo, r, c0, ep, sum, row_factor_deg(cur_end - cur_beg, mean));
        }
        a0 = float4_t{0.f, 0.f, 0.f, 0.f};
        a1 = float4_t{0.f, 0.f, 0.f, 0.f};
        before = false;
        do {  // next row; rows without entries are written on the way
          cur_beg = cur_end;
          ++r;
          cur_end = q1;
          q1 = q2;
          q2 = q3;
          q3 = r + 4 <= n ? rowptr[r + 4] : kEnd;
          if (cur_end == eu) write_empty(out, ldo, r, c0, ep);
        } while (cur_end == eu);
      }
      if (u & 1)
        fma4(a1, gg[u], vv[u]);
      else
        fma4(a0, gg[u], vv[u]);
    }
  }
  const float4_t sum = a0 + a1;
  if (cur_end == t) {
    if (before) {
      if (load_cols) *reinterpret_cast<float4_t*>(head + w * dpad + c0) = sum;
    } else {
      write_row(out, ldo, r, c0, ep, sum, row_factor_deg(cur_end - cur_beg, mean));
    }
    if (t == nnz)
      for (int64_t q = r + 1; q < n; ++q) write_empty(out, ldo, q, c0, ep);
    if (sub == 0 && blockIdx.y == 0) tail_row[w] = -1;
  } else if (before) {
    if (load_cols) *reinterpret_cast<float4_t*>(head + w * dpad + c0) = sum;
    if (sub == 0 && blockIdx.y == 0) tail_row[w] = -1;
  } else {
    if (load_cols) *reinterpret_cast<float4_t*>(tail + w * dpad + c0) = sum;
    if (sub == 0 && blockIdx.y == 0) tail_row[w] = (int32_t)r;
  }
}

template <typename T>
struct Gather;
template <>
struct Gather<_Float16> {
  __device__ static half4_t load(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
    return __builtin_bit_cast(half4_t, __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, 0));
  }
};
template <>
struct Gather<int16_t> {
  __device__ static short4_t load(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
    return __builtin_bit_cast(short4_t, __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, 0));
  }
};
template <>
struct Gather<int32_t> {
  __device__ static int4_t load(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
    return __builtin_bit_cast(int4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0));
  }
};
template <>
struct Gather<float> {
  __device__ static float4_t load(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
    return __builtin_bit_cast(float4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, 0));
  }
};

// The same aggregation with one worker per wave (layers wider than 128
// columns; each block row of the grid covers 256 columns).  All bookkeeping
// is wave-uniform and kept in 32-bit offsets from the chunk start:
//  - column indices and node scales arrive 64 edges at a time, one per lane,
//    two batches ahead (indices) and one batch ahead (scales), and are
//    broadcast with v_readlane;
//  - each gathered row is one buffer load whose row offset is a scalar
//    (one s_mul per edge) and whose column offset is a per-lane constant;
//  - the ends of the next 64 rows sit one per lane, double-buffered;
//  - U gathers are issued before the first is consumed.
// The byte size of C must fit in 32 bits (checked by the launcher).
template <typename T, int U>
__global__ __launch_bounds__(kBlock) void k_spmm_wave(
    int64_t n, int64_t nnz, const int64_t* __restrict__ rowptr,
    const int32_t* __restrict__ colidx, int mean, const float* __restrict__ g,
    const T* __restrict__ C, int32_t d, int64_t ldc,
    const float* __restrict__ alpha, const float* __restrict__ bias, int relu,
    float* __restrict__ out, int64_t ldo, int vec_out, int64_t chunk,
    int64_t workers, int32_t dpad, const int32_t* __restrict__ row_of,
    int32_t* __restrict__ tail_row, float* __restrict__ head,
    float* __restrict__ tail) {
  typedef typename Vec4<T>::type V;
  static_assert(64 % U == 0, "group size");
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
  if (w >= workers) return;
  const int c0 = blockIdx.y * 256 + lane * 4;
  const int64_t cl = c0 + 4 <= ldc ? c0 : ldc - 4;  // in-bounds load column
  Epi ep;
  ep.ncols = d - c0 < 0 ? 0 : (d - c0 > 4 ? 4 : d - c0);
  ep.relu = relu;
  ep.vec = vec_out != 0;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    ep.alpha[c] = c < ep.ncols ? alpha[c0 + c] : 0.f;
    ep.bias[c] = (c < ep.ncols && bias != nullptr) ? bias[c0 + c] : 0.f;
  }
  const bool own_cols = ep.ncols > 0;
  const int row_bytes = (int)(ldc * (int64_t)sizeof(T));
  const __amdgpu_buffer_rsrc_t rsC = raw_rsrc(C, (uint32_t)(n * row_bytes));
  const int voff = (int)(cl * (int64_t)sizeof(T));

  const int64_t s = w * chunk;
  const int nE = (int)((s + chunk < nnz ? s + chunk : nnz) - s);  // edges here
  const int64_t t = s + nE;
  // Row ends as offsets from s, clamped to [-1, chunk + 1].
  auto rel = [&](int64_t v) -> int {
    const int64_t x = v - s;
    return (int)(x < -1 ? -1 : (x > chunk + 1 ? chunk + 1 : x));
  };
  int64_t r = row_of[w];
  int64_t rbase = r;
  int win = rel(rowptr[rbase + 1 + lane < n ? rbase + 1 + lane : n]);
  int win_nx = rel(rowptr[rbase + 65 + lane < n ? rbase + 65 + lane : n]);
  const int64_t beg0 = rowptr[r];
  bool before = beg0 < s;
  int cur_beg = rel(beg0);
  int cur_end = __builtin_amdgcn_readlane(win, 0);
  if (!before) {
    for (int64_t q = r - 1; q >= 0 && rowptr[q] == s; --q)
      write_empty(out, ldo, q, c0, ep);
  }
  float4_t a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};

  // Batches of 64 edges: A = current (indices + scales), B = next (indices
  // + scales), Cn = the one after (indices only).
  auto ld_idx = [&](int eb) -> int32_t {
    const int x = eb + lane;
    return colidx[s + (x < nE ? x : nE - 1)];
  };
  int32_t jA = ld_idx(0);
  int32_t jB = ld_idx(64);
  float gA = g[jA];
  float gB = g[jB];
  int32_t jCn = ld_idx(128);

  for (int eb = 0; eb < nE; eb += 64) {
    for (int m = 0; m < 64; m += U) {
      const int e0 = eb + m;
      if (e0 >= nE) break;
      V vv[U];
      float gg[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = __builtin_amdgcn_readlane(jA, m + u);
        gg[u] = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                              __builtin_bit_cast(int, gA), m + u));
        vv[u] = Gather<T>::load(rsC, voff, (int)((uint32_t)j * (uint32_t)row_bytes));
      }
      if (e0 + U <= nE && cur_end >= e0 + U) {
        // No row ends inside this group: accumulate straight through.
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (u & 1)
            fma4(a1, gg[u], vv[u]);
          else
            fma4(a0, gg[u], vv[u]);
        }
        continue;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int eu = e0 + u;
        if (eu >= nE) break;
        if (eu == cur_end) {
          const float4_t sum = a0 + a1;
          if (before) {
            if (own_cols) *reinterpret_cast<float4_t*>(head + w * dpad + c0) = sum;
          } else if (own_cols) {
            write_row(out, ldo, r, c0, ep, sum, row_factor_deg(cur_end - cur_beg, mean));
          }
          a0 = float4_t{0.f, 0.f, 0.f, 0.f};
          a1 = float4_t{0.f, 0.f, 0.f, 0.f};
          before = false;
          do {  // next row; rows without entries are written on the way
            cur_beg = cur_end;
            ++r;
            if (r - rbase == 64) {
              rbase = r;
              win = win_nx;
              win_nx = rel(rowptr[rbase + 65 + lane < n ? rbase + 65 + lane : n]);
            }
            cur_end = __builtin_amdgcn_readlane(win, (int)(r - rbase));
            if (cur_end == eu && own_cols) write_empty(out, ldo, r, c0, ep);
          } while (cur_end == eu);
        }
        if (u & 1)
          fma4(a1, gg[u], vv[u]);
        else
          fma4(a0, gg[u], vv[u]);
      }
    }
    // Rotate the batches: A <- B, B <- (C, its scales), C <- next indices.
    jA = jB;
    gA = gB;
    jB = jCn;
    gB = g[jB];
    jCn = ld_idx(eb + 192);
  }
  const float4_t sum = a0 + a1;
  if (cur_end == nE) {
    if (before) {
      if (own_cols) *reinterpret_cast<float4_t*>(head + w * dpad + c0) = sum;
    } else if (own_cols) {
      write_row(out, ldo, r, c0, ep, sum, row_factor_deg(cur_end - cur_beg, mean));
    }
    if (t == nnz && own_cols)
      for (int64_t q = r + 1; q < n; ++q) write_empty(out, ldo, q, c0, ep);
    if (lane == 0 && blockIdx.y == 0) tail_row[w] = -1;
  } else if (before) {
    if (own_cols) *reinterpret_cast<float4_t*>(head + w * dpad + c0) = sum;
    if (lane == 0 && blockIdx.y == 0) tail_row[w] = -1;
  } else {
    if (own_cols) *reinterpret_cast<float4_t*>(tail + w * dpad + c0) = sum;
    if (lane == 0 && blockIdx.y == 0) tail_row[w] = (int32_t)r;
  }
}

// Lane views of the 8-bit layout (see k_bgemm_pop_q8): NB codes or NB exact
// halves per lane, widened to float4 with the unused components zero.
template <int NB>
__device__ inline uint32_t gather_codes(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
  if constexpr (NB == 4)
    return __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0);
  else if constexpr (NB == 2)
    return __builtin_amdgcn_raw_buffer_load_b16(rs, voff, soff, 0);
  else
    return __builtin_amdgcn_raw_buffer_load_b8(rs, voff, soff, 0);
}

template <int NB>
__device__ inline float4_t codes_to_float(uint32_t x) {
  float4_t f = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NB; ++c) f[c] = (float)(int)(int8_t)((x >> (8 * c)) & 0xff);
  return f;
}

// (dot - p) / 2 from a flagged row's exact products.
template <int NB>
__device__ inline float4_t gather_exact(__amdgpu_buffer_rsrc_t rs, int voff, int soff,
                                        float fpar) {
  float4_t v = {0.f, 0.f, 0.f, 0.f};
  if constexpr (NB == 4) {
    const half4_t x = __builtin_bit_cast(half4_t, __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, 0));
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = ((float)x[c] - fpar) * 0.5f;
  } else if constexpr (NB == 2) {
    const half2_t x = __builtin_bit_cast(half2_t, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0));
    v[0] = ((float)x[0] - fpar) * 0.5f;
    v[1] = ((float)x[1] - fpar) * 0.5f;
  } else {
    const _Float16 x = __builtin_bit_cast(_Float16, (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(rs, voff, soff, 0));
    v[0] = ((float)x - fpar) * 0.5f;
  }
  return v;
}

template <int NB>
__device__ inline void fma_n(float4_t& acc, float g, const float4_t& v) {
#pragma unroll
  for (int c = 0; c < NB; ++c) acc[c] = fmaf(v[c], g, acc[c]);
}

// Partial rows of the 8-bit path: NB floats per lane at p = base + NB*lane.
template <int NB>
__device__ inline void store_partial(float* p, const float4_t v) {
  if constexpr (NB == 4)
    *reinterpret_cast<float4_t*>(p) = v;
  else if constexpr (NB == 2)
    *reinterpret_cast<float2_t*>(p) = float2_t{v[0], v[1]};
  else
    *p = v[0];
}

template <int NB>
__device__ inline float4_t load_partial(const float* p) {
  float4_t v = {0.f, 0.f, 0.f, 0.f};
  if constexpr (NB == 4) {
    v = *reinterpret_cast<const float4_t*>(p);
  } else if constexpr (NB == 2) {
    const float2_t x = *reinterpret_cast<const float2_t*>(p);
    v[0] = x[0];
    v[1] = x[1];
  } else {
    v[0] = *p;
  }
  return v;
}

// What the aggregation does with a finished output row in the 8-bit path.
// Lane l holds columns l + 64c of the row (c < NB, interleaved).
//   NX == 0: write act(rowfac*alpha*acc + b) to out (columns l + 64c).
//   NX == 2: as 0, plus the self term of a two-weight GraphSAGE layer:
//            |g_r| * alpha_self[k] * Cself[r][k] (exact half products of the
//            node's own features with the self weights) before bias / act.
//   NX == 1: the next layer (K' = d inputs, d' <= 256 outputs, NBN bytes per
//            lane) is fused: its sign bits are the ballots of the output
//            values (word c = ballot of slot c, because lane l holds element
//            l + 64c), its scale is their mean magnitude (summed per lane
//            over c, then a butterfly: the order of the pack kernel), and its
//            products against the next weights (in LDS) are written as 8-bit
//            half-codes with the exact fallback, as k_bgemm_pop_q8 does.
// With NX == 1 the output row is also written to out if out != nullptr.
struct NextLayer {
  int32_t dn;          // next layer's output width d'
  int8_t* C8;          // codes [n][ldc8]
  int64_t ldc8;
  _Float16* C16;       // exact fallback rows [n][ldc16]
  int64_t ldc16;
  float* g;            // next layer's per-node scale
  int sym;             // fold D̂^-1/2 into the next scale
  const _Float16* Cself;  // NX == 2: self products [n][ldself], natural order
  int64_t ldself;
  const float* gself;     // NX == 2: per-node scale (its magnitude is β_i)
  const int32_t* slot;    // nullable: row r's next products / self products
                          // sit at row slot[r] (the source order), else at r
  const uint64_t* F;      // NX == 3: the layer's packed signs, row r at F + r ldF
  int64_t ldF;            // (r = slot[r] when slot is given)
  int32_t kin;            // NX == 3: the layer's input width
};

// The next layer's weights as finish_row reads them.
struct NextRegs {
  const uint64_t* sB;  // LDS: next weights, [kw'][NBN][64] interleaved columns
  uint64_t wr[4];      // or, when NB * NBN <= 4, this lane's words in registers:
                       // wr[w * NBN + c] = word w of column lane + 64c
};

// Everything finish_row reads besides a row's sums and the next weights:
// the first argument of the kernels that finish rows, so that it starts the
// kernel-argument segment.  finish_row reads it afresh at each call (scalar
// loads from that segment behind an opaque pointer, which the compiler
// cannot hoist) instead of the kernel holding its fields in scalar
// registers through the edge loop, where they would crowd out the loop's
// own values.  The per-column alpha, bias and alpha_self sit in LDS
// (stage_epi).
struct FinishArgs {
  NextLayer nx;
  float* out;            // [n][ldo]; nullable when a next layer is formed
  int64_t ldo;
  const float* alpha;    // this layer's alpha [d]
  const float* bias;     // [d] or null
  const float* alpha_s;  // two-weight layer: the self weights' alpha [d]
  int mean;              // destination factor, see row_factor_deg
  int relu;
  int32_t d;             // output width, at most 256
};

typedef const __attribute__((address_space(4))) FinishArgs* KernargFinish;
__device__ inline FinishArgs fresh_finish() {
#if defined(__HIP_DEVICE_COMPILE__)
  KernargFinish p = (KernargFinish)__builtin_amdgcn_kernarg_segment_ptr();
  __asm__ volatile("" : "+s"(p));
  return *p;
#else
  return FinishArgs{};  // (the host pass only parses device functions)
#endif
}

// LDS copy of alpha, bias and alpha_self (zero past d) for finish_row, one
// column per thread of the block; ends in a barrier.
__device__ inline void stage_epi(float (*s_epi)[256], const FinishArgs& fa) {
  static_assert(kBlock == 256, "one column per thread");
  const int t = threadIdx.x;
  const bool ok = t < fa.d;
  s_epi[0][t] = ok ? fa.alpha[t] : 0.f;
  s_epi[1][t] = ok && fa.bias != nullptr ? fa.bias[t] : 0.f;
  s_epi[2][t] = ok && fa.alpha_s != nullptr ? fa.alpha_s[t] : 0.f;
  __syncthreads();
}

// Without a fused next layer and with groups of 8 edges (short epilogues,
// frequent on graphs of short rows) the epilogue's arguments stay in the
// kernel's scalar registers and alpha, bias and alpha_self of a lane's
// columns in its registers: a kernel-argument read and LDS reads at every
// finished row measured slower there (arxiv-shaped, 123 -> 139-144 us), and
// these variants have the registers to spare.  finish_row's EPI_LDS says
// which form it takes.
template <int NB>
struct EpiRegs {
  float alpha[NB], bias[NB], alpha_s[NB];
};
template <int NB>
__device__ inline void make_epi_regs(EpiRegs<NB>& er, const FinishArgs& fa, int lane) {
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const int k = lane + 64 * c;
    const bool ok = k < fa.d;
    er.alpha[c] = ok ? fa.alpha[k] : 0.f;
    er.bias[c] = ok && fa.bias != nullptr ? fa.bias[k] : 0.f;
    er.alpha_s[c] = ok && fa.alpha_s != nullptr ? fa.alpha_s[k] : 0.f;
  }
}

// The first kw of a row's NW packed words (zero past kw), the row address
// the same in every lane: read-only, so they come through scalar loads.
template <int NW>
__device__ inline void load_row_words(uint64_t (&fw)[NW], const uint64_t* __restrict__ row,
                                      int kw) {
#pragma unroll
  for (int w = 0; w < NW; ++w) fw[w] = w < kw ? row[w] : 0ull;
}

template <int NX, int NB, int NBN, bool EPI_LDS>
__device__ inline void finish_row(int64_t r, int64_t deg, const float4_t acc,
                                  const float (*s_epi)[256], const EpiRegs<NB>& er,
                                  const NextRegs& nr, const FinishArgs& fa_arg, int lane) {
  // EPI_LDS: the arguments are read afresh (see FinishArgs) and alpha /
  // bias come from LDS; else from the kernel argument's scalar registers
  // and the lane's registers (EpiRegs).
  const FinishArgs fa = EPI_LDS ? fresh_finish() : fa_arg;
  const NextLayer& nx = fa.nx;
  bool valid[NB];  // column lane + 64c < d
#pragma unroll
  for (int c = 0; c < NB; ++c) valid[c] = lane + 64 * c < fa.d;
  const float rowfac = deg > 0 ? row_factor_deg(deg, fa.mean) : 0.f;
  int64_t dst = r;  // row of the next products / self products
  if (NX != 0 && nx.slot != nullptr) dst = nx.slot[r];
  float self[NB];
  if constexpr (NX == 3) {
    // The two-weight layer's self products, formed here: the row's own
    // packed signs (wave-uniform, scalar loads) against the self weights
    // staged in LDS (NBN words per lane and column) -- the products Cself
    // holds for NX == 2, exactly.
    const int kws = (nx.kin + 63) >> 6;  // <= NBN
    uint64_t fw[NBN];
    load_row_words<NBN>(fw, nx.F + dst * nx.ldF, kws);
    const float gi = fabsf(nx.gself[dst]);
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      uint32_t pc = 0;
#pragma unroll
      for (int w = 0; w < NBN; ++w) {
        if (w >= kws) continue;  // wave-uniform
        const uint64_t z = fw[w] ^ nr.sB[(w * NB + c) * 64 + lane];
        pc += __builtin_popcount((uint32_t)z);
        pc += __builtin_popcount((uint32_t)(z >> 32));
      }
      const int dot = nx.kin - 2 * (int)pc;
      self[c] = valid[c] ? gi * (EPI_LDS ? s_epi[2][lane + 64 * c] : er.alpha_s[c]) * (float)dot
                         : 0.f;
    }
  }
  if (NX == 2) {
    const float gi = fabsf(nx.gself[dst]);
#pragma unroll
    for (int c = 0; c < NB; ++c)
      self[c] = valid[c] ? gi * (EPI_LDS ? s_epi[2][lane + 64 * c] : er.alpha_s[c]) *
                               (float)nx.Cself[dst * nx.ldself + lane + 64 * c]
                         : 0.f;
  }
  float v[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const float al = EPI_LDS ? s_epi[0][lane + 64 * c] : er.alpha[c];
    const float bi = EPI_LDS ? s_epi[1][lane + 64 * c] : er.bias[c];
    float t = deg > 0 ? fmaf(acc[c], rowfac * al, bi) : bi;
    if (NX == 2 || NX == 3) t += self[c];
    v[c] = act(t, fa.relu);
  }
  if (NX != 1 || fa.out != nullptr) {
#pragma unroll
    for (int c = 0; c < NB; ++c)
      if (valid[c]) fa.out[r * fa.ldo + lane + 64 * c] = v[c];
  }
  if (NX != 1) return;
  // Next layer: signs (one ballot per 64 elements = one packed word) and
  // mean magnitude, exactly as the pack kernel forms them.
  uint64_t word[NB];
  float l1 = 0.f;
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    word[c] = __builtin_amdgcn_ballot_w64(valid[c] && v[c] >= 0.f);
    l1 += valid[c] ? fabsf(v[c]) : 0.f;
  }
  l1 = wave_sum(l1);
  float sc = l1 / (float)fa.d;
  if (nx.sym) sc = sc * (deg > 0 ? 1.0f / sqrtf((float)deg) : 0.f);
  const int kwn = (fa.d + 63) >> 6;  // <= NB
  const int Kn = fa.d;
  const int par = Kn & 1;
  bool big = false;
  uint32_t packed = 0;
  int dot[NBN];
#pragma unroll
  for (int c = 0; c < NBN; ++c) {
    uint32_t pc = 0;
#pragma unroll
    for (int w = 0; w < NB; ++w) {
      if (w >= kwn) break;
      const uint64_t bw = NB * NBN <= 4 ? nr.wr[(w * NBN + c) & 3]
                                        : nr.sB[(w * NBN + c) * 64 + lane];
      const uint64_t z = word[w] ^ bw;
      pc += __builtin_popcount((uint32_t)z);
      pc += __builtin_popcount((uint32_t)(z >> 32));
    }
    dot[c] = Kn - 2 * (int)pc;
    const int code = (dot[c] - par) >> 1;
    big |= (lane + 64 * c < nx.dn) && (code < -128 || code > 127);
    packed |= (uint32_t)(uint8_t)(int8_t)code << (8 * c);
  }
  store_codes<NBN>(nx.C8 + dst * nx.ldc8 + NBN * lane, packed);
  const bool flag = __builtin_amdgcn_ballot_w64(big) != 0;
  if (flag) store_exact<NBN>(nx.C16 + dst * nx.ldc16 + NBN * lane, dot);
  if (lane == 0) nx.g[dst] = flag ? -sc : sc;
}

// The next layer's weights for finish_row: in registers when a lane needs
// at most four words (NB * NBN <= 4; no LDS, no block barrier), else staged
// in LDS by the whole block (stage_weights, which ends in a barrier).
template <int NB, int NBN>
__device__ inline void load_next_weights(NextRegs& nx, int32_t dn, uint64_t* sBn,
                                         const uint64_t* __restrict__ Bn, int64_t ldbn,
                                         int32_t d, int lane) {
  const int kwn = (d + 63) >> 6;
  if constexpr (NB * NBN <= 4) {
#pragma unroll
    for (int w = 0; w < NB; ++w)
#pragma unroll
      for (int c = 0; c < NBN; ++c) {
        const int col = lane + 64 * c;
        nx.wr[(w * NBN + c) & 3] =
            (w < kwn && col < dn) ? Bn[(int64_t)col * ldbn + w] : 0ull;
      }
    nx.sB = nullptr;
  } else {
    stage_weights<NBN, true>(sBn, Bn, dn, ldbn, kwn, 0);
    nx.sB = sBn;
  }
}

// The row holding edge s, rowptr[r] <= s < rowptr[r+1] (rows without
// entries are skipped), by a wave-wide search: each step the 64 lanes probe
// 64 evenly spaced row starts of the current range [lo, hi), which shrinks
// 65-fold; once it is at most 64 rows wide, lane l loads the start and end
// of row lo + l.  Returns r; lo, and this lane's start / end, are the window
// the aggregation walks from.  Requires rowptr[0] <= s < rowptr[n].
__device__ inline int64_t find_row(const int64_t* __restrict__ rowptr, int64_t n, int64_t s,
                                   int lane, int64_t& lo_out, int64_t& start_l,
                                   int64_t& end_l) {
  int64_t lo = 0, hi = n;
  while (hi - lo > 64) {
    const int64_t step = (hi - lo + 64) / 65;
    const int64_t p = lo + (int64_t)(lane + 1) * step;
    const bool le = p < hi && rowptr[p] <= s;
    const int c = (int)__builtin_popcountll(__builtin_amdgcn_ballot_w64(le));
    const int64_t nhi = lo + (int64_t)(c + 1) * step;
    lo += (int64_t)c * step;
    if (nhi < hi) hi = nhi;
  }
  start_l = rowptr[lo + lane < n ? lo + lane : n];
  end_l = rowptr[lo + 1 + lane < n ? lo + 1 + lane : n];
  lo_out = lo;
  const uint64_t done = __builtin_amdgcn_ballot_w64(lo + 1 + lane <= n && end_l <= s);
  return lo + (int64_t)__builtin_popcountll(done);
}

__device__ inline int64_t readlane64(int64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Whole-wave aggregation over 8-bit half-codes (see k_bgemm_pop_q8):
//   sum_j g_j dot_jk = 2 * sum_j g_j code_jk + p * sum_j g_j.
// An edge whose source row is flagged (sign bit of g_j) reads that row's
// exact products from C16 instead and adds g_j (dot - p) / 2 to the same
// accumulator, so partial sums and the fix-up are the same as for exact
// storage.  Lane l accumulates columns l + 64c (c < NB); partial rows are
// stored in the same interleaved order.  Structure otherwise as
// k_spmm_wave, except that each wave finds its first row itself
// (find_row: no row plan is needed); finished rows go through
// finish_row<NX, NB, NBN>.  P = K mod 2 (the parity p): for even K the
// p * sum g term is zero and its running sum is not kept.
// Occupancy: 8 waves per SIMD for groups of 8 edges fusing the next layer's
// pack and GEMM, or the GraphSAGE self term for even K (their SGPRs then fit
// 8 waves; on the arxiv-shaped graph the forward pass measured 0.520 ->
// 0.500 ms, the GraphSAGE one 0.736 -> 0.712 ms, the products-shaped one
// within noise), else 6 (groups of 16, and the odd-K self term, spill in the
// edge loop at 8 waves).
template <int U, int NX, int NB, int NBN, int P>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(
    U == 8 && (NX == 1 || (NX == 3 && P == 0)) ? 8 : 6))) void k_spmm_wave_q8(
    FinishArgs fa, int64_t n, int64_t nnz, const int64_t* __restrict__ rowptr,
    const int32_t* __restrict__ colidx, const float* __restrict__ g,
    const int8_t* __restrict__ C8, int64_t ldc8, const _Float16* __restrict__ C16,
    int64_t ldc16, int par, int64_t chunk, int64_t workers, int32_t dpad,
    int32_t* __restrict__ tail_row, float* __restrict__ head,
    float* __restrict__ tail, const uint64_t* __restrict__ Bn, int64_t ldbn) {
  static_assert(64 % U == 0, "group size");
  extern __shared__ uint64_t sBn[];
  __shared__ float s_epi[3][256];
  // the scales of the window's 64 edges, read back as 16-byte broadcasts
  __shared__ __attribute__((aligned(16))) float s_gw[kWavesPerBlock][64];
  const int lane = threadIdx.x & 63;
  const int64_t wv = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
  const bool live = wv < workers;
  const int64_t w = live ? wv : workers - 1;  // waves past the end only stage
  const int64_t s = w * chunk;
  const int nE = (int)((s + chunk < nnz ? s + chunk : nnz) - s);
  const int64_t t = s + nE;
  auto ld_idx = [&](int eb) -> int32_t {
    const int x = eb + lane;
    return colidx[s + (x < nE ? x : nE - 1)];
  };
  int32_t jA = ld_idx(0);  // issued first: independent of everything else
  int32_t jB = ld_idx(64);
  NextRegs nr = {};
  if (NX == 1) load_next_weights<NB, NBN>(nr, fa.nx.dn, sBn, Bn, ldbn, fa.d, lane);
  // NX == 3: the self weights, NBN words by NB columns per lane, in LDS
  if (NX == 3) load_next_weights<NBN, NB>(nr, fa.d, sBn, Bn, ldbn, fa.nx.kin, lane);
  // where finish_row reads its arguments and alpha / bias (see EpiRegs)
  constexpr bool kEpiLds = NX == 1 || NX == 3 || U == 16;
  if constexpr (kEpiLds) stage_epi(s_epi, fa);
  EpiRegs<NB> er = {};
  if constexpr (!kEpiLds) make_epi_regs<NB>(er, fa, lane);
  if (!live) return;
  const int rb8 = (int)ldc8;
  const int rb16 = (int)(ldc16 * 2);
  const __amdgpu_buffer_rsrc_t rs8 = raw_rsrc(C8, (uint32_t)(n * rb8));
  const __amdgpu_buffer_rsrc_t rs16 = raw_rsrc(C16, (uint32_t)(n * rb16));
  const int voff8 = NB * lane;
  const int voff16 = 2 * NB * lane;
  const float fpar = (float)par;

  auto rel = [&](int64_t v) -> int {
    const int64_t x = v - s;
    return (int)(x < -1 ? -1 : (x > chunk + 1 ? chunk + 1 : x));
  };
  float gA = g[jA];
  int64_t rbase, start_l, end_l;
  int64_t r = find_row(rowptr, n, s, lane, rbase, start_l, end_l);
  int win = rel(end_l);
  int win_nx = rel(rowptr[rbase + 65 + lane < n ? rbase + 65 + lane : n]);
  const int64_t beg0 = readlane64(start_l, (int)(r - rbase));
  bool before = beg0 < s;
  int cur_beg = rel(beg0);
  int cur_end = __builtin_amdgcn_readlane(win, (int)(r - rbase));
  const float4_t zero4 = {0.f, 0.f, 0.f, 0.f};
  if (!before) {
    for (int64_t q = r - 1; q >= 0 && rowptr[q] == s; --q)
      finish_row<NX, NB, NBN, kEpiLds>(q, 0, zero4, s_epi, er, nr, fa, lane);
  }
  float4_t a0 = zero4, a1 = zero4;
  float gsum = 0.f;  // sum of g_j over the current row (for the parity term)
  float gB = g[jB];
  int32_t jCn = ld_idx(128);
  float* gw = &s_gw[wave_index_in_block()][0];
  for (int eb = 0; eb < nE; eb += 64) {
    const uint64_t flagged = __builtin_amdgcn_ballot_w64(__builtin_bit_cast(int, gA) < 0);
    gw[lane] = gA;
    for (int m = 0; m < 64; m += U) {
      const int e0 = eb + m;
      if (e0 >= nE) break;
      uint32_t vv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = __builtin_amdgcn_readlane(jA, m + u);
        vv[u] = gather_codes<NB>(rs8, voff8, (int)((uint32_t)j * (uint32_t)rb8));
      }
      const bool any_flag = ((flagged >> m) & ((1ull << U) - 1)) != 0;
      if (e0 + U <= nE && cur_end >= e0 + U && !any_flag) {
        // a group inside one row: its scales (the same in every lane) as
        // LDS broadcasts, whose latency hides behind the gathers
        float gg[U];
#pragma unroll
        for (int u = 0; u < U; u += 4) {
          const float4_t g4 = *reinterpret_cast<const float4_t*>(gw + m + u);
#pragma unroll
          for (int v = 0; v < 4; ++v) gg[u + v] = g4[v];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (u & 1)
            fma_n<NB>(a1, gg[u], codes_to_float<NB>(vv[u]));
          else
            fma_n<NB>(a0, gg[u], codes_to_float<NB>(vv[u]));
          if constexpr (P != 0) gsum += gg[u];
        }
        continue;
      }
      // A group with a row end or a flagged source, edge by edge (false once
      // past the chunk's end): unrolled for groups of 8, a loop for groups of
      // 16 (the body holds two row epilogues; their graphs have long rows and
      // few such groups, and 16 copies do not unroll).
      auto slow_edge = [&](int u) -> bool {
        const int eu = e0 + u;
        if (eu >= nE) return false;
        if (eu == cur_end) {
          const float4_t sum = P != 0 ? 2.f * (a0 + a1) + fpar * gsum : 2.f * (a0 + a1);
          if (before) {
            store_partial<NB>(head + w * dpad + NB * lane, sum);
          } else {
            finish_row<NX, NB, NBN, kEpiLds>(r, cur_end - cur_beg, sum, s_epi, er, nr, fa, lane);
          }
          a0 = zero4;
          a1 = zero4;
          gsum = 0.f;
          before = false;
          do {  // next row; rows without entries are finished on the way
            cur_beg = cur_end;
            ++r;
            if (r - rbase == 64) {
              rbase = r;
              win = win_nx;
              win_nx = rel(rowptr[rbase + 65 + lane < n ? rbase + 65 + lane : n]);
            }
            cur_end = __builtin_amdgcn_readlane(win, (int)(r - rbase));
            if (cur_end == eu)
              finish_row<NX, NB, NBN, kEpiLds>(r, 0, zero4, s_epi, er, nr, fa, lane);
          } while (cur_end == eu);
        }
        float gj = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                 __builtin_bit_cast(int, gA), m + u));
        float4_t v;
        if (__builtin_bit_cast(int, gj) < 0) {
          // Flagged source row: its exact products, as (dot - p) / 2.
          gj = fabsf(gj);
          const int j = __builtin_amdgcn_readlane(jA, m + u);
          v = gather_exact<NB>(rs16, voff16, (int)((uint32_t)j * (uint32_t)rb16), fpar);
        } else {
          v = codes_to_float<NB>(vv[u]);
        }
        if (u & 1)
          fma_n<NB>(a1, gj, v);
        else
          fma_n<NB>(a0, gj, v);
        if constexpr (P != 0) gsum += gj;
        return true;
      };
      static_assert(U == 8 || U == 16, "group sizes");
      if constexpr (U == 8) {
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (!slow_edge(u)) break;
      } else {
#pragma unroll 1
        for (int u = 0; u < U; ++u)
          if (!slow_edge(u)) break;
      }
    }
    jA = jB;
    gA = gB;
    jB = jCn;
    gB = g[jB];
    jCn = ld_idx(eb + 192);
  }
  const float4_t sum = P != 0 ? 2.f * (a0 + a1) + fpar * gsum : 2.f * (a0 + a1);
  if (cur_end == nE) {
    if (before) {
      store_partial<NB>(head + w * dpad + NB * lane, sum);
    } else {
      finish_row<NX, NB, NBN, kEpiLds>(r, cur_end - cur_beg, sum, s_epi, er, nr, fa, lane);
    }
    if (t == nnz)
      for (int64_t q = r + 1; q < n; ++q)
        finish_row<NX, NB, NBN, kEpiLds>(q, 0, zero4, s_epi, er, nr, fa, lane);
    if (lane == 0) tail_row[w] = -1;
  } else if (before) {
    store_partial<NB>(head + w * dpad + NB * lane, sum);
    if (lane == 0) tail_row[w] = -1;
  } else {
    store_partial<NB>(tail + w * dpad + NB * lane, sum);
    if (lane == 0) tail_row[w] = (int32_t)r;
  }
}

// Fix-up of the 8-bit path: rows cut by chunk boundaries, partial rows in
// interleaved order, finished with the same finish_row.  One wave serves
// four workers: their cut rows, row bounds and first two partial rows are
// loaded together (lanes 0..3 fetch the per-worker scalars), then the rows
// are finished in worker order.
template <int NX, int NB, int NBN>
__global__ __launch_bounds__(kBlock) void k_spmm_fix_q8(
    FinishArgs fa, const int64_t* __restrict__ rowptr, int64_t chunk, int64_t workers,
    int32_t dpad, const int32_t* __restrict__ tail_row,
    const float* __restrict__ head, const float* __restrict__ tail,
    const uint64_t* __restrict__ Bn, int64_t ldbn) {
  extern __shared__ uint64_t sBn[];
  __shared__ float s_epi[3][256];
  const int lane = threadIdx.x & 63;
  NextRegs nr = {};
  if (NX == 1) load_next_weights<NB, NBN>(nr, fa.nx.dn, sBn, Bn, ldbn, fa.d, lane);
  // NX == 3: the self weights, NBN words by NB columns per lane, in LDS
  if (NX == 3) load_next_weights<NBN, NB>(nr, fa.d, sBn, Bn, ldbn, fa.nx.kin, lane);
  constexpr bool kEpiLds = NX == 1 || NX == 3;  // where finish_row reads alpha / bias
  if constexpr (kEpiLds) stage_epi(s_epi, fa);
  EpiRegs<NB> er = {};
  if constexpr (!kEpiLds) make_epi_regs<NB>(er, fa, lane);
  const int64_t w0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block()) * 4;
  if (w0 >= workers) return;
  // lane q < 4: worker w0 + q's cut row and that row's bounds
  const int64_t wq = w0 + (lane & 3);
  const int32_t rq = wq < workers ? tail_row[wq] : -1;
  const int64_t bq = rq >= 0 ? rowptr[rq] : 0;
  const int64_t eq = rq >= 0 ? rowptr[rq + 1] : 0;
  float4_t acc[4], nxt[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {  // tail of the worker and the next head
    const int32_t r = __builtin_amdgcn_readlane(rq, q);
    if (r >= 0) {
      const int64_t w = w0 + q;
      acc[q] = load_partial<NB>(tail + w * dpad + NB * lane);
      nxt[q] = load_partial<NB>(head + (w + 1) * dpad + NB * lane);
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int32_t r = __builtin_amdgcn_readlane(rq, q);
    if (r < 0) continue;
    const int64_t w = w0 + q;
    const int64_t e = readlane64(eq, q);
    const int64_t wend = (e - 1) / chunk;  // > w: a cut row continues past w
    float4_t a = acc[q] + nxt[q];
    int64_t v = w + 2;
    for (; v + 8 <= wend + 1; v += 8) {  // eight loads in flight, added in order
      float4_t h[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) h[u] = load_partial<NB>(head + (v + u) * dpad + NB * lane);
#pragma unroll
      for (int u = 0; u < 8; ++u) a += h[u];
    }
    for (; v <= wend; ++v) a += load_partial<NB>(head + v * dpad + NB * lane);
    finish_row<NX, NB, NBN, kEpiLds>(r, e - readlane64(bq, q), a, s_epi, er, nr, fa, lane);
  }
}

// ------------------------------------------------ narrow 8-bit aggregation ----
//
// Layers of at most 64 output columns keep one code byte per column (column
// k at byte k of a 64-byte row).  In the k_spmm_wave_q8 layout a wave then
// spends one gather instruction per edge on one byte per lane.  Here a slot
// of G lanes covers a row's columns instead, CPL codes per lane (one 4-, 8-
// or 16-byte gather), so a wave works on S = 64 / G rows or edges at once.
//
// Work split: block b owns rows [b*R, b*R + R), R <= 64, and cuts their edge
// range into four equal shares, one per wave.  A wave takes the rows that
// start in its share and, as a partial, the row in progress where its share
// begins.  Rows are dealt to the slots in rounds of S.  In a round a row with
// at most kNarrowShort edges in the share is summed by its own slot, edge by
// edge in CSR order (row-parallel); a longer one by all slots together, slot
// q taking edges q, q + S, ... (edge-parallel), followed by a butterfly over
// the slots.  Complete rows are then finished by their slots in parallel.
// A row cut by a share boundary leaves its head pieces in LDS; after a
// block barrier the wave where it starts adds them, in share order, to the
// tail it holds in its slot.  A wave's last round of rows is finished after
// that barrier, together with its cut row, so the epilogue runs once per
// wave.  No atomics and no second kernel: the sums, and hence the results,
// do not depend on timing.
constexpr int kNarrowShort = 16;  // edges in a share up to which a row is row-parallel
// rows landed per lane and batch (1 KB of LDS per wave and row for 16-byte
// pieces, 256 B for 4-byte ones)
template <int CPL>
constexpr int narrow_batch() { return CPL == 4 ? 16 : 8; }

// Block barrier for data exchanged through LDS only: this wave's LDS
// operations complete first (lgkmcnt 0), while its global loads and stores
// may stay in flight (no vmcnt wait, unlike __syncthreads).
__device__ inline void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt 63, expcnt 7, lgkmcnt 0
  __builtin_amdgcn_s_barrier();
}

// 64-bit lane exchange within quads (DPP quad_perm control CTRL).
template <int CTRL>
__device__ inline uint64_t dpp_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, 0xF, 0xF, false);
  const uint32_t hi =
      (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, 0xF, 0xF, false);
  return ((uint64_t)hi << 32) | lo;
}

// Lane swaps between two registers: swap32 exchanges lanes 32..63 of a with
// lanes 0..31 of b; swap16 exchanges the odd 16-lane rows of a with the even
// rows of b.  (The results are read into scalars before the bit casts.)
__device__ inline void swap32(float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, a),
                                                  __builtin_bit_cast(uint32_t, b), false, false);
  const uint32_t x = r[0], y = r[1];
  a = __builtin_bit_cast(float, x);
  b = __builtin_bit_cast(float, y);
}
__device__ inline void swap16(float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, a),
                                                  __builtin_bit_cast(uint32_t, b), false, false);
  const uint32_t x = r[0], y = r[1];
  a = __builtin_bit_cast(float, x);
  b = __builtin_bit_cast(float, y);
}

// v[k] summed over the 64 / G lanes that share lane % G, the result in every
// lane, for CPL values per lane (CPL a multiple of 4; the whole wave active).
// A reduce-scatter first halves the values per lane twice (wave halves, then
// pairs of 16-lane rows: after it lane l holds value i + (CPL/4)(row & 1) +
// (CPL/2)(row >> 1) for i < CPL/4), the rows are then summed by rotations
// within the row, and the same two swaps bring every value back to every
// lane.  One swap or add per value and step instead of a lane exchange and
// an add per value for each of the six slot bits.
template <int G, int CPL>
__device__ inline void slot_allreduce(float (&v)[CPL]) {
  static_assert(CPL % 4 == 0, "values per lane");
  constexpr int H = CPL / 2, Q = CPL / 4;
  float h[H];
#pragma unroll
  for (int i = 0; i < H; ++i) {
    float a = v[i], b = v[i + H];
    swap32(a, b);
    h[i] = a + b;  // lanes 0..31: value i, lanes 32..63: value i + H
  }
  float p[Q];
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    float a = h[i], b = h[i + Q];
    swap16(a, b);
    p[i] = a + b;
  }
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    if constexpr (G <= 1) p[i] += dpp<0x121>(p[i]);  // row_ror:1
    if constexpr (G <= 2) p[i] += dpp<0x122>(p[i]);  // row_ror:2
    if constexpr (G <= 4) p[i] += dpp<0x124>(p[i]);  // row_ror:4
    p[i] += dpp<0x128>(p[i]);                        // row_ror:8
  }
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    float a = p[i], b = p[i];
    swap16(a, b);
    h[i] = a;
    h[i + Q] = b;
  }
#pragma unroll
  for (int i = 0; i < H; ++i) {
    float a = h[i], b = h[i];
    swap32(a, b);
    v[i] = a;
    v[i + H] = b;
  }
}

// One value per lane summed over the lanes that share lane % G, in every lane.
template <int G>
__device__ inline float slot_allreduce1(float t) {
  float a = t, b = t;
  swap32(a, b);
  t = a + b;
  a = t;
  b = t;
  swap16(a, b);
  t = a + b;
  if constexpr (G <= 1) t += dpp<0x121>(t);
  if constexpr (G <= 2) t += dpp<0x122>(t);
  if constexpr (G <= 4) t += dpp<0x124>(t);
  return t + dpp<0x128>(t);
}

// Gathered code rows land in LDS (buffer loads with the lds modifier: lane
// l's bytes go to base + size * l, a range past the buffer gives zeros), so
// a wave keeps NB rows per lane in flight without holding them in
// registers.  4-byte pieces for CPL == 4, else 16 bytes (CPL == 8 uses half).
typedef __attribute__((address_space(3))) void lds_void_t;
template <int CPL>
struct Landed {
  typedef typename std::conditional<CPL == 4, uint32_t, uint4>::type type;
  static constexpr int bytes = CPL == 4 ? 4 : 16;
};

// One landed piece per lane (wave-uniform LDS destination).
__device__ inline void land_piece16(__amdgpu_buffer_rsrc_t rs, void* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)lds, 16, voff, 0, 0, 0);
}
__device__ inline void land_piece4(__amdgpu_buffer_rsrc_t rs, void* lds, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)lds, 4, voff, 0, 0, 0);
}
template <int CPL, typename T>
__device__ inline void land_piece(__amdgpu_buffer_rsrc_t rs, T* lds, uint32_t voff) {
  if constexpr (CPL == 4)
    land_piece4(rs, (void*)lds, voff);
  else
    land_piece16(rs, (void*)lds, voff);
}

// Wait until this wave's landed rows are in LDS (vmcnt(0), other counters
// left alone), and keep the compiler from moving LDS reads above it.
__device__ inline void wait_landed() {
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __asm__ volatile("" ::: "memory");
}

__device__ inline float code_of(uint32_t w, int k) {
  return (float)(int)(int8_t)((w >> (8 * k)) & 0xff);
}

template <int CPL>
__device__ inline float landed_code(const typename Landed<CPL>::type& x, int k) {
  if constexpr (CPL == 4) {
    return code_of(x, k);
  } else {
    const uint32_t w = (k >> 2) == 0 ? x.x : (k >> 2) == 1 ? x.y : (k >> 2) == 2 ? x.z : x.w;
    return code_of(w, k & 3);
  }
}

// (dot - p) / 2 for CPL consecutive columns of a flagged row's exact products
// (halves; row offset voff bytes).
template <int CPL>
__device__ inline void gather_row_exact(float (&v)[CPL], __amdgpu_buffer_rsrc_t rs,
                                        uint32_t voff, float fpar) {
  // whole-vector bit casts (filling a local half array dword by dword has
  // been seen to compile into a single-dword load replicated across columns)
  if constexpr (CPL == 16) {
    const half8_t a = __builtin_bit_cast(half8_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                      rs, (int)voff, 0, 0));
    const half8_t b = __builtin_bit_cast(half8_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                      rs, (int)(voff + 16), 0, 0));
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      v[k] = ((float)a[k] - fpar) * 0.5f;
      v[8 + k] = ((float)b[k] - fpar) * 0.5f;
    }
  } else if constexpr (CPL == 8) {
    const half8_t a = __builtin_bit_cast(half8_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                      rs, (int)voff, 0, 0));
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = ((float)a[k] - fpar) * 0.5f;
  } else {
    const half4_t a = __builtin_bit_cast(half4_t, __builtin_amdgcn_raw_buffer_load_b64(
                                                      rs, (int)voff, 0, 0));
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = ((float)a[k] - fpar) * 0.5f;
  }
}

// One slot's batch of landed rows added to its sums: acc[k] += g_j code_jk
// and gs += g_j over the batch in edge order, where a flagged row (sign bit
// of g_j) counts with weight zero; then, only if the batch holds flagged rows,
// their exact products (dot - p) / 2 are added with weight |g_j|, again in
// edge order.  The fixed order keeps the sums reproducible.
template <int CPL, int NB>
__device__ inline void narrow_accumulate(float (&acc)[CPL], float& gs,
                                         const typename Landed<CPL>::type* base, int lane,
                                         const float (&gv)[NB], const uint32_t (&jv)[NB],
                                         __amdgpu_buffer_rsrc_t rs16, uint32_t rb16,
                                         uint32_t coff16, float fpar) {
  bool flagged = false;
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    const bool f = __builtin_bit_cast(int, gv[u]) < 0;
    flagged |= f;
    const float gj = f ? 0.f : gv[u];
    const typename Landed<CPL>::type x = base[u * 64 + lane];
#pragma unroll
    for (int k = 0; k < CPL; ++k) acc[k] = fmaf(landed_code<CPL>(x, k), gj, acc[k]);
    gs += gj;
  }
  if (__builtin_amdgcn_ballot_w64(flagged) == 0) return;
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    const bool f = __builtin_bit_cast(int, gv[u]) < 0;
    if (__builtin_amdgcn_ballot_w64(f) == 0) continue;
    if (f) {
      const float gj = fabsf(gv[u]);
      float v[CPL];
      gather_row_exact<CPL>(v, rs16, jv[u] * rb16 + coff16, fpar);
#pragma unroll
      for (int k = 0; k < CPL; ++k) acc[k] = fmaf(v[k], gj, acc[k]);
      gs += gj;
    }
    // one edge at a time, so the exact loads are not all hoisted (and held
    // in registers) ahead of the first
    __asm__ volatile("" ::: "memory");
  }
}

// Epilogue constants of the narrow layout: alpha, bias and (NX == 2) the self
// weights' alpha per column, staged in LDS by the block (zero past d); lane
// c of a slot reads columns CPL*c + k.
struct NarrowEpi {
  const float* s_alpha;  // LDS [3][64]: alpha, bias, alpha_self
  uint32_t valid;        // bit k: column CPL*c + k < d
  int relu;
  int32_t d;
  bool vec;              // out 16-byte aligned with ldo % 4 == 0
};

// A finished row in one slot: the same epilogue as finish_row (rescale,
// bias, self term, activation), the output written or, for NX == 1, the
// next layer formed in place.  Its scale is the mean |value| summed in the
// order of the pack kernel's wave reduction (lane c holds elements
// 16c .. 16c + 15, one 16-lane row of that reduction: a balanced tree inside
// the lane, then (row0 + row1) + (row2 + row3) across the slot), so fused and
// chained layers agree bit for bit.  With K' = d <= 64 every next product
// |dot| <= 64 fits an 8-bit half-code: no exact fallback is needed.
template <int G, int CPL, int NX>
__device__ inline void finish_slot(int64_t r, int64_t deg, int mean, const float (&sum)[CPL],
                                   const NarrowEpi& ep, int c, float* __restrict__ out,
                                   int64_t ldo, const NextLayer& nx, int nbn,
                                   const uint64_t* s_bn) {
  static_assert(CPL * G <= 64 && CPL <= 16 && CPL % 4 == 0, "narrow layout");
  const float rowfac = deg > 0 ? row_factor_deg(deg, mean) : 0.f;
  int64_t dst = r;  // row of the next products / self products
  if (NX != 0 && nx.slot != nullptr) dst = nx.slot[r];
  float gi = 0.f;
  if (NX == 2) gi = fabsf(nx.gself[dst]);
  // this lane's constants in 16-byte LDS reads, all issued before any use
  const float* al = ep.s_alpha + CPL * c;
  float av[CPL], bv[CPL], sv[NX == 2 ? CPL : 1];
#pragma unroll
  for (int k = 0; k < CPL; k += 4) {
    const float4_t a4 = *reinterpret_cast<const float4_t*>(al + k);
    const float4_t b4 = *reinterpret_cast<const float4_t*>(al + 64 + k);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      av[k + u] = a4[u];
      bv[k + u] = b4[u];
    }
    if constexpr (NX == 2) {
      const float4_t s4 = *reinterpret_cast<const float4_t*>(al + 128 + k);
#pragma unroll
      for (int u = 0; u < 4; ++u) sv[k + u] = s4[u];
    }
  }
  float v[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) {
    const bool ok = (ep.valid >> k) & 1;
    float t = deg > 0 ? fmaf(sum[k], rowfac * av[k], bv[k]) : bv[k];
    if (NX == 2)
      t += ok ? gi * sv[k] * (float)nx.Cself[dst * nx.ldself + CPL * c + k] : 0.f;
    v[k] = act(t, ep.relu);
  }
  if (NX != 1 || out != nullptr) {
    float* o = out + r * ldo + CPL * c;
    if (ep.vec && ep.valid == (1u << CPL) - 1) {
#pragma unroll
      for (int k = 0; k < CPL; k += 4) {
        float4_t q4;
#pragma unroll
        for (int u = 0; u < 4; ++u) q4[u] = v[k + u];
        *reinterpret_cast<float4_t*>(o + k) = q4;
      }
    } else {
#pragma unroll
      for (int k = 0; k < CPL; ++k)
        if ((ep.valid >> k) & 1) o[k] = v[k];
    }
  }
  if (NX != 1) return;
  uint32_t m = 0;
  float a[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const bool ok = k < CPL && ((ep.valid >> k) & 1);
    if (k < CPL) m |= (uint32_t)(ok && v[k] >= 0.f) << k;
    a[k] = ok ? fabsf(v[k < CPL ? k : 0]) : 0.f;
  }
  // the slot's G lanes are one quad or part of one: DPP quad exchanges
  uint64_t word = (uint64_t)m << (CPL * c);
  if (G >= 2) word |= dpp_u64<0xB1>(word);  // quad_perm [1,0,3,2]: lane ^ 1
  if (G >= 4) word |= dpp_u64<0x4E>(word);  // quad_perm [2,3,0,1]: lane ^ 2
  float qd[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    qd[i] = (a[4 * i] + a[4 * i + 1]) + (a[4 * i + 2] + a[4 * i + 3]);
  float l1 = (qd[0] + qd[1]) + (qd[2] + qd[3]);
  if (G >= 2) l1 = l1 + dpp<0xB1>(l1);
  if (G >= 4) l1 = l1 + dpp<0x4E>(l1);
  float sc = l1 / (float)ep.d;
  if (nx.sym) {
    // D-hat^-1/2 of this row: the symmetric row factor itself when this
    // layer is symmetric too
    const float isd =
        mean == 0 ? rowfac : (deg > 0 ? 1.0f / sqrtf((float)deg) : 0.f);
    sc = sc * isd;
  }
  const int Kn = ep.d;
  const int par = Kn & 1;
  for (int kq = c; kq < nx.dn; kq += G) {
    const uint64_t z = word ^ s_bn[kq];
    const int pc = __builtin_popcount((uint32_t)z) + __builtin_popcount((uint32_t)(z >> 32));
    const int code = ((Kn - 2 * pc) - par) >> 1;
    nx.C8[dst * nx.ldc8 + nbn * (kq & 63) + (kq >> 6)] = (int8_t)code;
  }
  if (c == 0) nx.g[dst] = sc;
}

template <int G, int CPL, int NX>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void k_spmm_narrow(
    int64_t n, const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    int mean, const float* __restrict__ g, const int8_t* __restrict__ C8, int64_t ldc8,
    const _Float16* __restrict__ C16, int64_t ldc16, int par, int32_t d,
    const float* __restrict__ alpha, const float* __restrict__ bias, int relu,
    float* __restrict__ out, int64_t ldo, int32_t rpb, NextLayer nx, int nbn,
    const uint64_t* __restrict__ Bn, int64_t ldbn, const float* __restrict__ alpha_s) {
  constexpr int S = 64 / G;
  extern __shared__ uint64_t s_bn[];  // NX == 1: word 0 of each next weight column
  __shared__ float s_head[kWavesPerBlock][64];  // the piece of a row cut at a share's start
  __shared__ __attribute__((aligned(16))) float s_epi[3][64];  // alpha, bias, alpha_self
  // A chunk of CH edges lands in LDS through NLI instructions of EPI = 64 / G
  // edges each (lane l: edge EPI i + l / G, bytes CPL (l % G) ..); chunk edge
  // k's piece c sits at landed index G k + c, its scale at s_gk[k].
  constexpr int EPI = 64 / G;
  constexpr int NLI = G == 4 ? 8 : 4;
  constexpr int CH = NLI * EPI;
  constexpr int JR = CH / 64;
  typedef typename Landed<CPL>::type LandT;
  __shared__ LandT s_land[kWavesPerBlock][NLI * 64];
  __shared__ float s_gk[kWavesPerBlock][CH];
  const int lane = threadIdx.x & 63;
  const int wv = wave_index_in_block();
  const int q = lane / G;
  const int c = lane % G;
  const int64_t r_lo = (int64_t)blockIdx.x * rpb;
  const int nr = (int)(n - r_lo < rpb ? n - r_lo : rpb);
  // lane l < nr: bounds of row r_lo + l (lanes past nr repeat the last row)
  const int64_t rl = r_lo + (lane < nr ? lane : nr - 1);
  int64_t st, en;
  {
    // The block's constants and the row bounds, every load issued before
    // the first LDS store:
    // thread t < 64 fetches column t's alpha, bias and alpha_self (zero past
    // d, the byte ranges ending there), and with NX == 1 thread t < d' word
    // 0 of next weight column t (d' <= 256 threads).
    const int t = threadIdx.x;
    const uint32_t eo = t < 64 ? (uint32_t)t * 4u : kPastEnd;
    const uint32_t eb4 = (uint32_t)d * 4u;
    const float e_al = __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(raw_rsrc(alpha, eb4), (int)eo, 0, 0));
    const float e_bi = __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(raw_rsrc(bias, bias != nullptr ? eb4 : 0u),
                                                    (int)eo, 0, 0));
    float e_as = 0.f;
    if constexpr (NX == 2)
      e_as = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(raw_rsrc(alpha_s, eb4), (int)eo, 0, 0));
    uint64_t e_bn = 0;
    if constexpr (NX == 1)
      e_bn = __builtin_bit_cast(
          uint64_t, __builtin_amdgcn_raw_buffer_load_b64(
                        raw_rsrc(Bn, (uint32_t)(nx.dn * ldbn * 8)),
                        (int)(t < nx.dn ? (uint32_t)(t * ldbn) * 8u : kPastEnd), 0, 0));
    st = rowptr[rl];
    en = rowptr[rl + 1];
    if (t < 64) {
      s_epi[0][t] = e_al;
      s_epi[1][t] = e_bi;
      s_epi[2][t] = e_as;
    }
    if (NX == 1 && t < nx.dn) s_bn[t] = e_bn;
  }
  NarrowEpi ep;
  ep.s_alpha = &s_epi[0][0];
  ep.relu = relu;
  ep.d = d;
  ep.vec = ((uintptr_t)out & 15) == 0 && (ldo & 3) == 0;
  ep.valid = 0;
#pragma unroll
  for (int k = 0; k < CPL; ++k) ep.valid |= (uint32_t)(CPL * c + k < d) << k;
  const int64_t eb = readlane64(st, 0);
  const int64_t ee = readlane64(en, nr - 1);
  const int total = (int)(ee - eb);
  const bool last = wv == kWavesPerBlock - 1;
  const int rs_l = (int)(st - eb);
  const int re_l = (int)(en - eb);
  // Share boundaries bnd[0..4] (relative edge positions, nondecreasing):
  // each share takes an equal part of the edges still unassigned, except
  // that a share whose rows (the row cut at its start and those starting in
  // it) would number more than S ends at the start of the row that would be
  // its (S+1)-th, saving its wave a second round of rows, as long as the
  // shares after it then stay within one landing chunk of the equal split.
  const int L = (total + kWavesPerBlock - 1) / kWavesPerBlock;
  int bnd[kWavesPerBlock + 1];
  bnd[0] = 0;
  bnd[kWavesPerBlock] = total;
#pragma unroll
  for (int i = 1; i < kWavesPerBlock; ++i) {
    const int lo = bnd[i - 1];
    const int rem = kWavesPerBlock - i + 1;  // shares left, this one included
    int b = lo + (total - lo + rem - 1) / rem;
    const int first =
        (int)__builtin_popcountll(__builtin_amdgcn_ballot_w64(lane < nr && rs_l < lo));
    const int cut = (first > 0 && __builtin_amdgcn_readlane(re_l, first - 1) > lo) ? 1 : 0;
    const int ends =
        (int)__builtin_popcountll(__builtin_amdgcn_ballot_w64(lane < nr && rs_l < b));
    if (ends - first + cut > S) {
      const int bc = __builtin_amdgcn_readlane(rs_l, first + S - cut);
      if (total - bc <= (rem - 1) * (L + CH)) b = bc;
    }
    bnd[i] = b;
  }
  int ws = 0, we = total;  // bnd[wv], bnd[wv + 1]
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    if (i == wv) ws = bnd[i];
    if (i == wv + 1) we = bnd[i];
  }
  const int o_b = (int)__builtin_popcountll(__builtin_amdgcn_ballot_w64(lane < nr && rs_l < ws));
  const int o_e = last ? nr
                       : (int)__builtin_popcountll(
                             __builtin_amdgcn_ballot_w64(lane < nr && rs_l < we));
  int h = o_b;
  if (o_b > 0 && __builtin_amdgcn_readlane(re_l, o_b - 1) > ws) h = o_b - 1;
  const float fpar = (float)par;
  const uint32_t rb8 = (uint32_t)ldc8;
  const uint32_t rb16 = (uint32_t)(ldc16 * 2);
  const uint32_t coff8 = (uint32_t)(CPL * c);
  const uint32_t coff16 = (uint32_t)(2 * CPL * c);
  const __amdgpu_buffer_rsrc_t rs8 = raw_rsrc(C8, (uint32_t)(n * (int64_t)rb8));
  const __amdgpu_buffer_rsrc_t rs16 = raw_rsrc(C16, (uint32_t)(n * (int64_t)rb16));
  const __amdgpu_buffer_rsrc_t rsi = raw_rsrc(colidx + eb, (uint32_t)total * 4u);
  const __amdgpu_buffer_rsrc_t rsg = raw_rsrc(g, (uint32_t)(n * 4));
  // The first round's first batch of edge indices is requested before the
  // block barrier (its range is the one the round loop computes for base h).
  uint32_t jpre[JR];
#pragma unroll
  for (int r = 0; r < JR; ++r) jpre[r] = 0;
  if (h < o_e) {
    const int p0 = max(__builtin_amdgcn_readlane(rs_l, h), ws);
    const int p1 = min(__builtin_amdgcn_readlane(re_l, min(h + S, o_e) - 1), we);
#pragma unroll
    for (int r = 0; r < JR; ++r)
      jpre[r] = __builtin_amdgcn_raw_buffer_load_b32(
          rsi, (int)(p0 + 64 * r + lane < p1 ? (uint32_t)(p0 + 64 * r + lane) * 4u : kPastEnd),
          0, 0);
  }
  lds_barrier();  // s_epi and s_bn are read by finish_slot

  LandT* land = &s_land[wv][0];
  float* sgk = &s_gk[wv][0];
  // Lands chunk edges [0, nk) whose indices lane l holds in jr[r] (edge
  // 64 r + l): their scales into sgk, their code pieces into land; issued()
  // runs once the loads are in flight, before the wait.
  auto land_chunk = [&](const uint32_t (&jr)[JR], int nk, auto&& issued) {
    float gk[JR];
#pragma unroll
    for (int r = 0; r < JR; ++r)
      gk[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                            rsg, (int)(64 * r + lane < nk ? jr[r] * 4u : kPastEnd),
                                            0, 0));
    // every lane exchange first, so their latencies overlap; then the loads
    uint32_t lo[NLI];
#pragma unroll
    for (int i = 0; i < NLI; ++i) {
      const int k = EPI * i + lane / G;
      const uint32_t j = (uint32_t)__shfl((int)jr[(EPI * i) / 64], (EPI * i) % 64 + lane / G);
      lo[i] = k < nk ? j * rb8 + coff8 : kPastEnd;
    }
#pragma unroll
    for (int i = 0; i < NLI; ++i) {
      if (EPI * i >= nk) break;  // wave-uniform
      land_piece<CPL>(rs8, land + i * 64, lo[i]);
    }
    issued();
    wait_landed();
#pragma unroll
    for (int r = 0; r < JR; ++r)
      if (64 * r < nk) sgk[64 * r + lane] = gk[r];
  };
  // Adds chunk edges k[u] (those with ok[u]) to a slot's sums, in order u =
  // 0..3; all four LDS reads are issued before the first is used.  A flagged
  // source row (sign bit of g) adds its exact products instead, its index
  // read back from colidx at byte offset ipos[u].
  auto add_edges4 = [&](float (&a)[CPL], float& sg, const int (&k)[4], const bool (&ok)[4],
                        const uint32_t (&ipos)[4]) {
    LandT x[4];
    float gv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      x[u] = land[G * k[u] + c];
      gv[u] = ok[u] ? sgk[k[u]] : 0.f;
    }
    bool any = false;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool f = __builtin_bit_cast(int, gv[u]) < 0;
      any |= f;
      const float gw = f ? 0.f : gv[u];
#pragma unroll
      for (int kk = 0; kk < CPL; ++kk) a[kk] = fmaf(landed_code<CPL>(x[u], kk), gw, a[kk]);
      sg += gw;
    }
    if (__builtin_amdgcn_ballot_w64(any) == 0) return;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool f = __builtin_bit_cast(int, gv[u]) < 0;
      if (__builtin_amdgcn_ballot_w64(f) == 0) continue;
      if (f) {
        const uint32_t j = __builtin_amdgcn_raw_buffer_load_b32(rsi, (int)ipos[u], 0, 0);
        float v[CPL];
        gather_row_exact<CPL>(v, rs16, j * rb16 + coff16, fpar);
        const float ga = fabsf(gv[u]);
#pragma unroll
        for (int kk = 0; kk < CPL; ++kk) a[kk] = fmaf(v[kk], ga, a[kk]);
        sg += ga;
      }
      __asm__ volatile("" ::: "memory");
    }
  };
  // The last round's rows are finished after the block barrier, together
  // with the row cut at this share's end (its pieces from the following
  // waves added into its slot): one epilogue for them all.  Their sums wait
  // in this wave's landing buffer (idle by then; CPL floats per lane fit).
  static_assert(64 * CPL * 4 <= NLI * 64 * (int)sizeof(LandT), "sums fit the landing buffer");
  float* keep_lds = reinterpret_cast<float*>(&s_land[wv][0]) + CPL * lane;
  bool keep_fin = false, keep_tail = false;
  int64_t keep_row = 0;
  int keep_rs = 0, keep_re = 0;
  for (int base = h; base < o_e; base += S) {
    const int idx = base + q;
    const bool on = idx < o_e;
    const int ix = on ? idx : base;
    const int rs = __shfl(rs_l, ix);
    const int re = __shfl(re_l, ix);
    const int cb = rs > ws ? rs : ws;
    const int ce = re < we ? re : we;
    const int len = (on && ce > cb) ? ce - cb : 0;
    const bool lng = len > kNarrowShort;
    float acc[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) acc[k] = 0.f;
    float gs = 0.f;
    // The round's rows own one contiguous edge range [r0, r1) (within the
    // share); it lands chunk by chunk, every lane of a landing busy, the next
    // chunk's indices loading while this one lands.  Short rows then walk
    // their own edges in LDS (row-parallel); each long row is summed
    // edge-parallel per chunk (slot q on edges q, q + S, ..., then a
    // butterfly) and its owner adds the chunk totals in chunk order.
    const int nrow = min(S, o_e - base);
    const int r0 = __builtin_amdgcn_readfirstlane(cb);
    const int r1 = __builtin_amdgcn_readlane(ce, (nrow - 1) * G);
    uint32_t jn[JR];
    if (base == h) {
#pragma unroll
      for (int r = 0; r < JR; ++r) jn[r] = jpre[r];
    } else {
#pragma unroll
      for (int r = 0; r < JR; ++r)
        jn[r] = __builtin_amdgcn_raw_buffer_load_b32(
            rsi, (int)(r0 + 64 * r + lane < r1 ? (uint32_t)(r0 + 64 * r + lane) * 4u : kPastEnd),
            0, 0);
    }
    // running strided sums of the long row in progress (it may continue
    // into the next chunk: rows are contiguous, so at most one does)
    float tmp[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) tmp[k] = 0.f;
    float tg = 0.f;
    for (int cbase = r0; cbase < r1; cbase += CH) {
      const int nk = min(CH, r1 - cbase);
      uint32_t jr[JR];
#pragma unroll
      for (int r = 0; r < JR; ++r) jr[r] = jn[r];
      land_chunk(jr, nk, [&]() {
#pragma unroll
        for (int r = 0; r < JR; ++r) {
          const int e = cbase + CH + 64 * r + lane;
          jn[r] = __builtin_amdgcn_raw_buffer_load_b32(
              rsi, (int)(e < r1 ? (uint32_t)e * 4u : kPastEnd), 0, 0);
        }
      });
      const int a0 = max(cb, cbase);
      const int a1 = min(ce, cbase + nk);
      const int cnt = (on && a1 > a0) ? a1 - a0 : 0;
      {
        // short rows: batches of four edges while any slot has edges left
        // (at most kNarrowShort per row in this chunk)
        const int sc = lng ? 0 : cnt;
        for (int t = 0; t < kNarrowShort; t += 4) {
          if (__builtin_amdgcn_ballot_w64(sc > t) == 0) break;
          int k[4];
          bool ok[4];
          uint32_t ip[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            ok[u] = !lng && t + u < cnt;
            k[u] = ok[u] ? a0 + t + u - cbase : 0;
            ip[u] = (uint32_t)(a0 + t + u) * 4u;
          }
          add_edges4(acc, gs, k, ok, ip);
        }
      }
      uint64_t lm = __builtin_amdgcn_ballot_w64(c == 0 && lng && cnt > 0);
      while (lm != 0) {
        const int ld = (int)__builtin_ctzll(lm);
        lm &= lm - 1;
        const int la = __builtin_amdgcn_readlane(a0, ld) - cbase;
        const int ln = __builtin_amdgcn_readlane(cnt, ld);
        const int mt = (ln + S - 1) / S;
        for (int t = 0; t < mt; t += 4) {
          int k[4];
          bool ok[4];
          uint32_t ip[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int kq = q + S * (t + u);
            ok[u] = kq < ln;
            k[u] = ok[u] ? la + kq : 0;
            ip[u] = (uint32_t)(cbase + la + kq) * 4u;
          }
          add_edges4(tmp, tg, k, ok, ip);
        }
        if (__builtin_amdgcn_readlane(ce, ld) <= cbase + nk) {  // the row ends here
          slot_allreduce<G, CPL>(tmp);
          // the sum of g is used for odd K only (fpar = 0 otherwise)
          if (par != 0) tg = slot_allreduce1<G>(tg);
          if (q == ld / G) {
#pragma unroll
            for (int k = 0; k < CPL; ++k) acc[k] = tmp[k];
            gs = tg;
          }
#pragma unroll
          for (int k = 0; k < CPL; ++k) tmp[k] = 0.f;
          tg = 0.f;
        }
      }
    }
    float sum[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) sum[k] = 2.f * acc[k] + fpar * gs;
    const bool headp = on && rs < ws;
    const bool tailp = on && !headp && re > we;
    if (headp) {
#pragma unroll
      for (int k = 0; k < CPL; ++k) s_head[wv][CPL * c + k] = sum[k];
    }
    const bool fin = on && !headp && !tailp;
    if (base + S < o_e) {
      if (fin)
        finish_slot<G, CPL, NX>(r_lo + idx, re - rs, mean, sum, ep, c, out, ldo, nx, nbn,
                                s_bn);
    } else {
#pragma unroll
      for (int k = 0; k < CPL; ++k) keep_lds[k] = sum[k];
      keep_fin = fin || tailp;
      keep_tail = tailp;
      keep_row = r_lo + idx;
      keep_rs = rs;
      keep_re = re;
    }
  }
  lds_barrier();
  float keep[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) keep[k] = keep_lds[k];
  // The row this wave started that runs past its share (the tail slot of
  // the last round): the heads of the waves whose shares start inside it,
  // added in share order.
  if (keep_tail) {
    int kend = wv;
#pragma unroll
    for (int m = 1; m < kWavesPerBlock; ++m)
      if (m > wv && bnd[m] < keep_re) kend = m;
    for (int m = wv + 1; m <= kend; ++m) {
#pragma unroll
      for (int k = 0; k < CPL; ++k) keep[k] += s_head[m][CPL * c + k];
    }
  }
  if (__builtin_amdgcn_ballot_w64(keep_fin) != 0 && keep_fin)
    finish_slot<G, CPL, NX>(keep_row, keep_re - keep_rs, mean, keep, ep, c, out, ldo, nx, nbn,
                            s_bn);
}

// Rows cut by chunk boundaries: tail of the owning worker, then the heads of
// the following workers, added in order.  A group of LC lanes (LC a power of
// two covering the layer width, at most 64) serves one worker, so every cut
// row is combined in parallel.
template <int LC>
__global__ __launch_bounds__(kBlock) void k_spmm_fix(
    const int64_t* __restrict__ rowptr, int mean, int32_t d,
    const float* __restrict__ alpha, const float* __restrict__ bias, int relu,
    float* __restrict__ out, int64_t ldo, int64_t chunk, int64_t workers,
    int32_t dpad, const int32_t* __restrict__ tail_row,
    const float* __restrict__ head, const float* __restrict__ tail) {
  const int lane = threadIdx.x & 63;
  const int64_t w = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / LC;
  if (w >= workers) return;
  const int sub = lane % LC;
  const int32_t r = tail_row[w];
  if (r < 0) return;
  const int64_t wend = (rowptr[r + 1] - 1) / chunk;
  const float rowfac = row_factor(rowptr, r, mean);
  for (int k = sub; k < d; k += LC) {
    float sacc = tail[w * dpad + k];
    int64_t v = w + 1;
    for (; v + 8 <= wend + 1; v += 8) {  // eight loads in flight, added in order
      float h[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) h[u] = head[(v + u) * dpad + k];
#pragma unroll
      for (int u = 0; u < 8; ++u) sacc += h[u];
    }
    for (; v <= wend; ++v) sacc += head[v * dpad + k];
    const float b = bias != nullptr ? bias[k] : 0.f;
    out[(int64_t)r * ldo + k] = act(fmaf(sacc, rowfac * alpha[k], b), relu);
  }
}

hipError_t launch_fix(const int64_t* rowptr, int mean, int32_t d, const float* alpha,
                      const float* bias, int relu, float* out, int64_t ldo,
                      const SpmmPlan& p, const int32_t* tail_row, const float* head,
                      const float* tail, hipStream_t stream) {
  const int lc = d <= 4 ? 4 : d <= 8 ? 8 : d <= 16 ? 16 : d <= 32 ? 32 : 64;
  const int64_t threads = p.workers * lc;
  const dim3 grid((unsigned)((threads + kBlock - 1) / kBlock));
#define BIGCN_FIX(LCV)                                                          \
  hipLaunchKernelGGL(k_spmm_fix<LCV>, grid, dim3(kBlock), 0, stream, rowptr, mean, d, \
                     alpha, bias, relu, out, ldo, p.chunk, p.workers, p.dpad,      \
                     tail_row, head, tail)
  switch (lc) {
    case 4: BIGCN_FIX(4); break;
    case 8: BIGCN_FIX(8); break;
    case 16: BIGCN_FIX(16); break;
    case 32: BIGCN_FIX(32); break;
    default: BIGCN_FIX(64); break;
  }
#undef BIGCN_FIX
  return hipGetLastError();
}

// row_of[w] = the row holding edge w*chunk.  One thread per row.
__global__ __launch_bounds__(kBlock) void k_spmm_rows(
    int64_t n, const int64_t* __restrict__ rowptr, int64_t chunk,
    int32_t* __restrict__ row_of) {
  const int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (r >= n) return;
  const int64_t a = rowptr[r], b = rowptr[r + 1];
  if (b <= a) return;
  for (int64_t w = (a + chunk - 1) / chunk; w * chunk < b; ++w) row_of[w] = (int32_t)r;
}

// Two-weight GraphSAGE layer on a graph without edges: every row is its
// self term, act(b_k + |g_i| alpha_self[k] Cself[i][k]).
__global__ __launch_bounds__(kBlock) void k_sage_self_only(
    int64_t n, int32_t d, const float* __restrict__ g, const _Float16* __restrict__ Cself,
    int64_t ldself, const float* __restrict__ alpha_s, const float* __restrict__ bias,
    int relu, float* __restrict__ out, int64_t ldo) {
  const int64_t idx = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (idx >= n * (int64_t)d) return;
  const int64_t i = idx / d;
  const int k = (int)(idx - i * d);
  const float self = fabsf(g[i]) * alpha_s[k] * (float)Cself[i * ldself + k];
  const float t = (bias != nullptr ? bias[k] : 0.f) + self;
  out[i * ldo + k] = act(t, relu);
}

// Graph without edges: every row is act(bias).
__global__ __launch_bounds__(kBlock) void k_spmm_empty(
    int64_t n, int32_t d, const float* __restrict__ bias, int relu,
    float* __restrict__ out, int64_t ldo) {
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= n * (int64_t)d) return;
  const int64_t r = i / d;
  const int k = (int)(i - r * d);
  out[r * ldo + k] = act(bias != nullptr ? bias[k] : 0.f, relu);
}

inline unsigned grid_cap(int64_t want, int64_t cap) {
  if (want < 1) want = 1;
  return (unsigned)(want < cap ? want : cap);
}

template <int CN, typename T>
hipError_t bgemm_pop_typed(const uint64_t* F, int64_t M, int64_t ldf,
                           const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                           T* C, int64_t ldc, int vec, hipStream_t stream) {
  constexpr int RM = 4;
  const int kw = (K + 63) >> 6;
  const size_t lds = (size_t)kw * CN * 64 * sizeof(uint64_t);
  const int64_t tiles = (M + RM - 1) / RM;
  dim3 grid(grid_cap((tiles + kWavesPerBlock - 1) / kWavesPerBlock, 4096),
            (unsigned)((N + 64 * CN - 1) / (64 * CN)));
  hipLaunchKernelGGL((k_bgemm_pop<CN, RM, T>), grid, dim3(kBlock), lds, stream,
                     F, M, ldf, B, N, ldb, K, C, ldc, vec);
  return hipGetLastError();
}

template <int CN>
hipError_t bgemm_pop_cn(const uint64_t* F, int64_t M, int64_t ldf,
                        const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                        void* C, IType ct, int64_t ldc, hipStream_t stream) {
  const size_t es = itype_size(ct);
  const int vec = (ldc % CN == 0) && ((uintptr_t)C % (CN * es) == 0);
  switch (ct) {
    case IType::F16:
      return bgemm_pop_typed<CN>(F, M, ldf, B, N, ldb, K, (_Float16*)C, ldc, vec, stream);
    case IType::I16:
      return bgemm_pop_typed<CN>(F, M, ldf, B, N, ldb, K, (int16_t*)C, ldc, vec, stream);
    default:
      return bgemm_pop_typed<CN>(F, M, ldf, B, N, ldb, K, (int32_t*)C, ldc, vec, stream);
  }
}

template <int L, typename T>
hipError_t spmm_typed(int64_t n, int64_t nnz, const int64_t* rowptr,
                      const int32_t* colidx, int mean, const float* g,
                      const T* C, int32_t d, int64_t ldc, const float* alpha,
                      const float* bias, int relu, float* out, int64_t ldo,
                      const SpmmPlan& p, void* ws, hipStream_t stream) {
  char* base = (char*)ws;
  const int32_t* row_of = (const int32_t*)(base + p.off_rowof);
  int32_t* tail_row = (int32_t*)(base + p.off_tailrow);
  float* head = (float*)(base + p.off_head);
  float* tail = (float*)(base + p.off_tail);
  constexpr int P = 64 / L;
  constexpr int U = 8;  // edges per group; one group in flight ahead
  const int vec_out = (ldo % 4 == 0) && ((uintptr_t)out % 16 == 0);
  const int64_t waves = (p.workers + P - 1) / P;
  dim3 grid((unsigned)((waves + kWavesPerBlock - 1) / kWavesPerBlock),
            (unsigned)((d + L * 4 - 1) / (L * 4)));
  hipLaunchKernelGGL((k_spmm<L, T, U>), grid, dim3(kBlock), 0, stream, n, nnz,
                     rowptr, colidx, mean, g, C, d, ldc, alpha, bias, relu, out,
                     ldo, vec_out, p.chunk, p.workers, p.dpad, row_of, tail_row,
                     head, tail);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_fix(rowptr, mean, d, alpha, bias, relu, out, ldo, p, tail_row, head,
                    tail, stream);
}

template <typename T>
hipError_t spmm_wave_typed(int64_t n, int64_t nnz, const int64_t* rowptr,
                           const int32_t* colidx, int mean, const float* g,
                           const T* C, int32_t d, int64_t ldc, const float* alpha,
                           const float* bias, int relu, float* out, int64_t ldo,
                           const SpmmPlan& p, void* ws, hipStream_t stream) {
  char* base = (char*)ws;
  const int32_t* row_of = (const int32_t*)(base + p.off_rowof);
  int32_t* tail_row = (int32_t*)(base + p.off_tailrow);
  float* head = (float*)(base + p.off_head);
  float* tail = (float*)(base + p.off_tail);
  const int vec_out = (ldo % 4 == 0) && ((uintptr_t)out % 16 == 0);
  dim3 grid((unsigned)((p.workers + kWavesPerBlock - 1) / kWavesPerBlock),
            (unsigned)((d + 255) / 256));
  constexpr int U = 8;
  hipLaunchKernelGGL((k_spmm_wave<T, U>), grid, dim3(kBlock), 0, stream, n, nnz,
                     rowptr, colidx, mean, g, C, d, ldc, alpha, bias, relu, out,
                     ldo, vec_out, p.chunk, p.workers, p.dpad, row_of, tail_row,
                     head, tail);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_fix(rowptr, mean, d, alpha, bias, relu, out, ldo, p, tail_row, head,
                    tail, stream);
}

// Lanes per worker for a layer width: 4 columns per lane; wider than 128
// columns takes whole-wave workers (L = 64).
inline int spmm_lanes(int32_t d) {
  const int lanes = (d + 3) / 4;
  return lanes <= 2 ? 2 : lanes <= 4 ? 4 : lanes <= 8 ? 8 : lanes <= 12 ? 12
       : lanes <= 16 ? 16 : lanes <= 32 ? 32 : 64;
}

template <typename T>
hipError_t spmm_dispatch_l(int64_t n, int64_t nnz, const int64_t* rowptr,
                           const int32_t* colidx, int mean, const float* g,
                           const T* C, int32_t d, int64_t ldc,
                           const float* alpha, const float* bias, int relu,
                           float* out, int64_t ldo, const SpmmPlan& p, void* ws,
                           hipStream_t stream) {
#define BIGCN_SPMM_L(LV)                                                       \
  return spmm_typed<LV, T>(n, nnz, rowptr, colidx, mean, g, C, d, ldc, alpha, \
                           bias, relu, out, ldo, p, ws, stream)
  switch (spmm_lanes(d)) {
    case 2: BIGCN_SPMM_L(2);
    case 4: BIGCN_SPMM_L(4);
    case 8: BIGCN_SPMM_L(8);
    case 12: BIGCN_SPMM_L(12);
    case 16: BIGCN_SPMM_L(16);
    case 32: BIGCN_SPMM_L(32);
    default:
      // Whole-wave workers address C with 32-bit buffer offsets.
      if ((uint64_t)n * (uint64_t)ldc * sizeof(T) > 0xFFFFFFFFull) BIGCN_SPMM_L(32);
      return spmm_wave_typed<T>(n, nnz, rowptr, colidx, mean, g, C, d, ldc, alpha,
                                bias, relu, out, ldo, p, ws, stream);
  }
#undef BIGCN_SPMM_L
}

// Fused binary GEMM of the FQ variant (unused otherwise).
struct PackQ8 {
  const int32_t* slot = nullptr;  // output row order (nullable)
  const uint64_t* B = nullptr;
  int32_t N = 0;
  int64_t ldb = 0;
  int8_t* C8 = nullptr;
  int64_t ldc8 = 0;
  _Float16* C16 = nullptr;
  int64_t ldc16 = 0;
};

template <bool STD, int RW, int KWT, int NBQ>
hipError_t pack_rows_launch(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                            const float* mu, const float* rstd, const int64_t* rowptr,
                            int sym, uint64_t* bits, int64_t ldw, float* scale,
                            const PackQ8& pq, hipStream_t stream) {
  const int64_t groups = (rows + RW - 1) / RW;
  // The fused GEMM's waves each load their weight words (and the column
  // statistics): with one column per lane fewer waves, taking several row
  // groups each, measured faster (500 inputs, 64 outputs: 10.3 us at 1024
  // blocks, 12.4 us at 2465); with 2 or 4 columns per lane a row costs more
  // ALU work and the full 8192 blocks measured faster (products-shaped
  // layer 0, 100 inputs and 256 outputs: about 0.08 ms less than at 1024).
  dim3 grid(grid_cap((groups + kWavesPerBlock - 1) / kWavesPerBlock, NBQ == 1 ? 1024 : 8192));
  const size_t lds = (STD && KWT > 16) ? (size_t)2 * cols * sizeof(float) : 0;
  hipLaunchKernelGGL((k_pack_rows<STD, RW, KWT, NBQ>), grid, dim3(kBlock), lds, stream, x,
                     rows, cols, ldx, mu, rstd, rowptr, sym, bits, ldw, scale, pq.B, pq.N,
                     pq.ldb, pq.C8, pq.ldc8, pq.C16, pq.ldc16, pq.slot);
  return hipGetLastError();
}

template <bool STD, int NBQ = 0>
hipError_t pack_rows_dispatch(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                              const float* mu, const float* rstd, const int64_t* rowptr,
                              int sym, uint64_t* bits, int64_t ldw, float* scale,
                              hipStream_t stream, const PackQ8& pq = PackQ8()) {
  const int kw = (cols + 63) >> 6;
#define BIGCN_PACK(RWV, KWV)                                                               \
  return pack_rows_launch<STD, RWV, KWV, NBQ>(x, rows, cols, ldx, mu, rstd, rowptr, sym, \
                                              bits, ldw, scale, pq, stream)
  if (kw <= 1) BIGCN_PACK(8, 1);
  if (kw <= 2) BIGCN_PACK(8, 2);
  if (kw <= 4) BIGCN_PACK(4, 4);
  if constexpr (NBQ <= 2) {
    if (kw <= 8) BIGCN_PACK(2, 8);
  }
  if constexpr (NBQ <= 1) {
    if (kw <= 16) BIGCN_PACK(1, 16);
  }
  if constexpr (NBQ == 0) BIGCN_PACK(1, 32);
  // the fused GEMM keeps at most 16 weight words per lane
  return hipErrorInvalidValue;
#undef BIGCN_PACK
}

}  // namespace

// ------------------------------------------------------------- launchers ----

hipError_t launch_pack(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                       const float* mu, const float* rstd,
                       const int64_t* rowptr, int sym, uint64_t* bits,
                       int64_t ldw, float* scale, hipStream_t stream, const int32_t* slot) {
  if (rows == 0) return hipSuccess;
  const int kw = (cols + 63) >> 6;
  // k_pack_rows writes a group's words with one lane per word (RW * ldw <=
  // 64 for the RW its dispatch picks from kw)
  const int rw = kw <= 2 ? 8 : kw <= 4 ? 4 : kw <= 8 ? 2 : 1;
  if (kw <= 32 && ldx <= kPackRowsMaxLd && rw * ldw <= 64) {
    PackQ8 pq;
    pq.slot = slot;
    if (mu != nullptr)
      return pack_rows_dispatch<true>(x, rows, cols, ldx, mu, rstd, rowptr, sym, bits,
                                      ldw, scale, stream, pq);
    return pack_rows_dispatch<false>(x, rows, cols, ldx, mu, rstd, rowptr, sym, bits,
                                     ldw, scale, stream, pq);
  }
  dim3 grid(grid_cap((rows + kWavesPerBlock - 1) / kWavesPerBlock, 8192));
  if (mu != nullptr)
    hipLaunchKernelGGL(k_pack<true>, grid, dim3(kBlock), 0, stream, x, rows, cols,
                       ldx, mu, rstd, rowptr, sym, bits, ldw, scale, slot);
  else
    hipLaunchKernelGGL(k_pack<false>, grid, dim3(kBlock), 0, stream, x, rows,
                       cols, ldx, mu, rstd, rowptr, sym, bits, ldw, scale, slot);
  return hipGetLastError();
}

// A lane keeps the weight words of its NB columns in registers, at most 16:
// inputs of more words would keep them in LDS inside a loop the compiler
// does not unroll; there the separate pack and GEMM are faster (1433 inputs,
// 64 outputs: 15.1 us fused against 8.0 + 5.2 us).
bool pack_bgemm_q8_supported(int32_t cols, int32_t N, int64_t ldx) {
  if (cols < 1 || N < 1 || N > 256 || ldx < cols || ldx > kPackRowsMaxLd) return false;
  return (int64_t)((cols + 63) / 64) * q8_lane_bytes(N) <= 16;
}

hipError_t launch_pack_bgemm_q8(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                                const float* mu, const float* rstd, const int64_t* rowptr,
                                int sym, const uint64_t* B, int32_t N, int64_t ldb,
                                int8_t* C8, int64_t ldc8, void* C16, int64_t ldc16,
                                float* g, hipStream_t stream, const int32_t* slot) {
  if (rows == 0) return hipSuccess;
  PackQ8 pq;
  pq.slot = slot;
  pq.B = B;
  pq.N = N;
  pq.ldb = ldb;
  pq.C8 = C8;
  pq.ldc8 = ldc8;
  pq.C16 = (_Float16*)C16;
  pq.ldc16 = ldc16;
#define BIGCN_PQ(NBV)                                                                    \
  return mu != nullptr ? pack_rows_dispatch<true, NBV>(x, rows, cols, ldx, mu, rstd, rowptr, \
                                                       sym, nullptr, 0, g, stream, pq)       \
                       : pack_rows_dispatch<false, NBV>(x, rows, cols, ldx, mu, rstd, rowptr, \
                                                        sym, nullptr, 0, g, stream, pq)
  switch (q8_lane_bytes(N)) {
    case 1: BIGCN_PQ(1);
    case 2: BIGCN_PQ(2);
    default: BIGCN_PQ(4);
  }
#undef BIGCN_PQ
}

hipError_t launch_bgemm_popcount(const uint64_t* F, int64_t M, int64_t ldf,
                                 const uint64_t* B, int32_t N, int64_t ldb,
                                 int32_t K, void* C, IType ct, int64_t ldc,
                                 hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int kw = (K + 63) >> 6;
  // Columns per lane: as many as the width needs (up to 4), limited so the
  // packed weight slab stays within 64 KiB of LDS.
  int cn = N <= 64 ? 1 : (N <= 128 ? 2 : 4);
  while (cn > 1 && (size_t)kw * cn * 64 * 8 > 65536) cn >>= 1;
  if (cn == 4) return bgemm_pop_cn<4>(F, M, ldf, B, N, ldb, K, C, ct, ldc, stream);
  if (cn == 2) return bgemm_pop_cn<2>(F, M, ldf, B, N, ldb, K, C, ct, ldc, stream);
  return bgemm_pop_cn<1>(F, M, ldf, B, N, ldb, K, C, ct, ldc, stream);
}

SpmmPlan spmm_plan(int64_t n, int64_t nnz, int32_t d, int64_t max_workers) {
  (void)n;
  SpmmPlan p;
  // About 16K workers on big graphs; chunks of 16 .. 2048 edges.
  int64_t chunk = 16;
  while (chunk < 2048 && chunk * 2 * 16384 <= nnz) chunk *= 2;
  if (max_workers >= 1 && (nnz + chunk - 1) / chunk > max_workers)
    chunk = (nnz + max_workers - 1) / max_workers;
  p.chunk = chunk;
  p.workers = nnz > 0 ? (nnz + chunk - 1) / chunk : 1;
  const int64_t slab = 4 * spmm_lanes(d);
  // Wide enough for both partial-row layouts: L lanes x 4 columns (exact
  // products) and 64 lanes x NB columns (8-bit path).
  p.dpad = (int32_t)std::max<int64_t>(((d + slab - 1) / slab) * slab,
                                      64 * q8_lane_bytes(d));
  auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
  size_t off = 0;
  p.off_rowof = off;
  off += up((size_t)p.workers * 4);
  p.off_tailrow = off;
  off += up((size_t)p.workers * 4);
  p.off_head = off;
  off += up((size_t)p.workers * p.dpad * 4);
  p.off_tail = off;
  off += up((size_t)p.workers * p.dpad * 4);
  p.bytes = off;
  return p;
}

hipError_t launch_spmm_rows(int64_t n, int64_t nnz, const int64_t* rowptr,
                            const SpmmPlan& plan, void* workspace,
                            hipStream_t stream) {
  if (nnz == 0 || n == 0) return hipSuccess;
  int32_t* row_of = (int32_t*)((char*)workspace + plan.off_rowof);
  hipLaunchKernelGGL(k_spmm_rows, dim3((unsigned)((n + kBlock - 1) / kBlock)),
                     dim3(kBlock), 0, stream, n, rowptr, plan.chunk, row_of);
  return hipGetLastError();
}

hipError_t launch_spmm(int64_t n, int64_t nnz, const int64_t* rowptr,
                       const int32_t* colidx, int mean, const float* g,
                       const void* C, IType ct, int32_t d, int64_t ldc,
                       const float* alpha, const float* bias, int relu,
                       float* out, int64_t ldo, const SpmmPlan& plan,
                       void* workspace, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  if (nnz == 0) {
    const int64_t total = n * (int64_t)d;
    hipLaunchKernelGGL(k_spmm_empty, dim3((unsigned)((total + kBlock - 1) / kBlock)),
                       dim3(kBlock), 0, stream, n, d, bias, relu, out, ldo);
    return hipGetLastError();
  }
  switch (ct) {
    case IType::F16:
      return spmm_dispatch_l<_Float16>(n, nnz, rowptr, colidx, mean, g,
                                       (const _Float16*)C, d, ldc, alpha, bias,
                                       relu, out, ldo, plan, workspace, stream);
    case IType::I16:
      return spmm_dispatch_l<int16_t>(n, nnz, rowptr, colidx, mean, g,
                                      (const int16_t*)C, d, ldc, alpha, bias,
                                      relu, out, ldo, plan, workspace, stream);
    case IType::F32:
      return spmm_dispatch_l<float>(n, nnz, rowptr, colidx, mean, g, (const float*)C, d,
                                    ldc, alpha, bias, relu, out, ldo, plan, workspace,
                                    stream);
    default:
      return spmm_dispatch_l<int32_t>(n, nnz, rowptr, colidx, mean, g,
                                      (const int32_t*)C, d, ldc, alpha, bias,
                                      relu, out, ldo, plan, workspace, stream);
  }
}

bool q8_supported(int64_t n, int32_t N, int32_t K) {
  if (N < 1 || N > 256 || K < 1 || K > 2048) return false;
  const uint64_t row = 64u * (uint64_t)q8_lane_bytes(N);
  return (uint64_t)n * row <= 0xFFFFFFFFull && (uint64_t)n * row * 2u <= 0xFFFFFFFFull;
}

hipError_t launch_bgemm_q8(const uint64_t* F, int64_t M, int64_t ldf,
                           const uint64_t* B, int32_t N, int64_t ldb, int32_t K,
                           int8_t* C8, int64_t ldc8, void* C16, int64_t ldc16,
                           float* g, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  constexpr int RM = 4;
  const int nb = q8_lane_bytes(N);
  const int kw = (K + 63) >> 6;
  const size_t lds = (size_t)kw * nb * 64 * sizeof(uint64_t);
  const int64_t tiles = (M + RM - 1) / RM;
  dim3 grid(grid_cap((tiles + kWavesPerBlock - 1) / kWavesPerBlock, 4096));
#define BIGCN_Q8G(NBV)                                                                  \
  hipLaunchKernelGGL((k_bgemm_pop_q8<RM, NBV>), grid, dim3(kBlock), lds, stream, F, M, \
                     ldf, B, N, ldb, K, C8, ldc8, (_Float16*)C16, ldc16, g)
  switch (nb) {
    case 1: BIGCN_Q8G(1); break;
    case 2: BIGCN_Q8G(2); break;
    default: BIGCN_Q8G(4); break;
  }
#undef BIGCN_Q8G
  return hipGetLastError();
}

template <int NX, int NB, int NBN>
hipError_t spmm_q8_nx(int64_t n, int64_t nnz, const int64_t* rowptr,
                      const int32_t* colidx, int mean, const float* g,
                      const int8_t* C8, int64_t ldc8, const void* C16, int64_t ldc16,
                      int32_t K, int32_t d, const float* alpha, const float* bias,
                      int relu, float* out, int64_t ldo, const SpmmPlan& p, void* ws,
                      const FusedNext& fn, hipStream_t stream) {
  char* base = (char*)ws;
  int32_t* tail_row = (int32_t*)(base + p.off_tailrow);
  float* head = (float*)(base + p.off_head);
  float* tail = (float*)(base + p.off_tail);
  FinishArgs fa;
  NextLayer& nx = fa.nx;
  nx.dn = fn.d_out;
  nx.C8 = fn.C8;
  nx.ldc8 = fn.ldc8;
  nx.C16 = (_Float16*)fn.C16;
  nx.ldc16 = fn.ldc16;
  nx.g = fn.g;
  nx.sym = !mean;
  nx.slot = fn.slot;
  nx.Cself = (const _Float16*)fn.Cself;
  nx.ldself = fn.ldself;
  nx.gself = g;
  nx.F = fn.F;
  nx.ldF = fn.ldF;
  nx.kin = fn.kin;
  fa.out = out;
  fa.ldo = ldo;
  fa.alpha = alpha;
  fa.bias = bias;
  fa.alpha_s = fn.alpha_self;
  fa.mean = mean;
  fa.relu = relu;
  fa.d = d;
  // LDS for the weights finish_row multiplies with: the next layer's (NX 1,
  // when a lane needs more than four words) or the self weights (NX 3)
  const size_t lds = NX == 3 ? (size_t)((fn.kin + 63) >> 6) * NB * 64 * sizeof(uint64_t)
                     : (NX > 0 && NB * NBN > 4)
                         ? (size_t)((d + 63) >> 6) * NBN * 64 * sizeof(uint64_t) : 0;
  const uint64_t* wB = NX == 3 ? fn.wself : fn.wbits;
  const int64_t ldB = NX == 3 ? fn.ldw_self : fn.ldw;
  dim3 grid((unsigned)((p.workers + kWavesPerBlock - 1) / kWavesPerBlock));
  // Gathers in flight per wave: groups of 16 edges where rows average at
  // least 64 entries (a group then almost always lies inside one row, and
  // more gathers in flight measured faster: reddit-shaped forward, 492
  // entries per row, 3.95 -> 3.77 ms), else 8 (shorter rows cut more groups,
  // which then take the edge-by-edge path: arxiv-shaped forward, 14 entries
  // per row, 3 % slower at 16; products-shaped, 52 per row, unchanged).
  auto launch = [&](auto u, auto par) {
    constexpr int UV = decltype(u)::value, PV = decltype(par)::value;
    hipLaunchKernelGGL((k_spmm_wave_q8<UV, NX, NB, NBN, PV>), grid, dim3(kBlock), lds, stream,
                       fa, n, nnz, rowptr, colidx, g, C8, ldc8, (const _Float16*)C16, ldc16,
                       PV, p.chunk, p.workers, p.dpad, tail_row, head, tail, wB, ldB);
  };
  using I8 = std::integral_constant<int, 8>;
  using I16 = std::integral_constant<int, 16>;
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  // (the self term formed in the epilogue keeps groups of 8: at 16 it would
  // not fit the register budget; so do layers of at most 64 columns, which
  // come here only for graphs of 2^31 entries or more: their 16-edge loop
  // indexed its codes through scratch memory)
  bool long_rows = nnz >= 64 * n;
  if constexpr (NX != 3 && NB >= 2) {
    if (long_rows) {
      if (K & 1) launch(I16{}, P1{}); else launch(I16{}, P0{});
    }
  } else {
    long_rows = false;
  }
  if (!long_rows) {
    if (K & 1) launch(I8{}, P1{}); else launch(I8{}, P0{});
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t fix_waves = (p.workers + 3) / 4;
  hipLaunchKernelGGL((k_spmm_fix_q8<NX, NB, NBN>),
                     dim3((unsigned)((fix_waves + kWavesPerBlock - 1) / kWavesPerBlock)),
                     dim3(kBlock), lds, stream, fa, rowptr, p.chunk, p.workers, p.dpad,
                     tail_row, head, tail, wB, ldB);
  return hipGetLastError();
}

template <int NB>
hipError_t spmm_q8_nb(int64_t n, int64_t nnz, const int64_t* rowptr,
                      const int32_t* colidx, int mean, const float* g,
                      const int8_t* C8, int64_t ldc8, const void* C16, int64_t ldc16,
                      int32_t K, int32_t d, const float* alpha, const float* bias,
                      int relu, float* out, int64_t ldo, const SpmmPlan& p, void* ws,
                      const FusedNext& fn, hipStream_t stream) {
#define BIGCN_Q8S(NX, NBN)                                                               \
  return spmm_q8_nx<NX, NB, NBN>(n, nnz, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, \
                                 K, d, alpha, bias, relu, out, ldo, p, ws, fn, stream)
  if (fn.kind == 0) BIGCN_Q8S(0, 1);
  if (fn.kind == 2) BIGCN_Q8S(2, 1);
  if constexpr (NB >= 2) {
    if (fn.kind == 3) BIGCN_Q8S(3, 16 / NB);  // NBN: the self weights' words per lane
  }
  switch (q8_lane_bytes(fn.d_out)) {
    case 1: BIGCN_Q8S(1, 1);
    case 2: BIGCN_Q8S(1, 2);
    default: BIGCN_Q8S(1, 4);
  }
#undef BIGCN_Q8S
}

// Rows per block of the narrow aggregation, at most one per lane of the
// block's row window: n / 800, within [8, 64] (measured: 8 for 2.7 K rows,
// 24 for 20 K rows, 64 for 169 K rows beat their neighbours).
int32_t narrow_rows_per_block(int64_t n) {
  const int64_t r = n / 800;
  return (int32_t)(r < 8 ? 8 : r > 64 ? 64 : r);
}

template <int G, int CPL>
hipError_t spmm_narrow_gc(int64_t n, const int64_t* rowptr, const int32_t* colidx,
                          int mean, const float* g, const int8_t* C8, int64_t ldc8,
                          const void* C16, int64_t ldc16, int32_t K, int32_t d,
                          const float* alpha, const float* bias, int relu, float* out,
                          int64_t ldo, const FusedNext& fn, hipStream_t stream) {
  NextLayer nx = {};
  nx.dn = fn.d_out;
  nx.C8 = fn.C8;
  nx.ldc8 = fn.ldc8;
  nx.C16 = (_Float16*)fn.C16;
  nx.ldc16 = fn.ldc16;
  nx.g = fn.g;
  nx.sym = !mean;
  nx.slot = fn.slot;
  nx.Cself = (const _Float16*)fn.Cself;
  nx.ldself = fn.ldself;
  nx.gself = g;
  const int32_t rpb = narrow_rows_per_block(n);
  const dim3 grid((unsigned)((n + rpb - 1) / rpb));
  const int nbn = fn.kind == 1 ? q8_lane_bytes(fn.d_out) : 1;
  // one thread per next weight column stages its first word
  if (fn.kind == 1 && fn.d_out > kBlock) return hipErrorInvalidValue;
  const size_t lds = fn.kind == 1 ? (size_t)fn.d_out * sizeof(uint64_t) : 0;
#define BIGCN_NARROW(NX)                                                                   \
  hipLaunchKernelGGL((k_spmm_narrow<G, CPL, NX>), grid, dim3(kBlock), lds, stream, n,      \
                     rowptr, colidx, mean, g, C8, ldc8, (const _Float16*)C16, ldc16, K & 1, \
                     d, alpha, bias, relu, out, ldo, rpb, nx, nbn, fn.wbits, fn.ldw,        \
                     fn.alpha_self)
  switch (fn.kind) {
    case 1: BIGCN_NARROW(1); break;
    case 2: BIGCN_NARROW(2); break;
    default: BIGCN_NARROW(0); break;
  }
#undef BIGCN_NARROW
  return hipGetLastError();
}

// Layers of at most 64 columns: lanes per slot and codes per lane by width.
hipError_t spmm_narrow(int64_t n, const int64_t* rowptr, const int32_t* colidx, int mean,
                       const float* g, const int8_t* C8, int64_t ldc8, const void* C16,
                       int64_t ldc16, int32_t K, int32_t d, const float* alpha,
                       const float* bias, int relu, float* out, int64_t ldo,
                       const FusedNext& fn, hipStream_t stream) {
  if (d <= 4)
    return spmm_narrow_gc<1, 4>(n, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                                alpha, bias, relu, out, ldo, fn, stream);
  if (d <= 8)
    return spmm_narrow_gc<1, 8>(n, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                                alpha, bias, relu, out, ldo, fn, stream);
  if (d <= 16)
    return spmm_narrow_gc<1, 16>(n, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                                 alpha, bias, relu, out, ldo, fn, stream);
  if (d <= 32)
    return spmm_narrow_gc<2, 16>(n, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                                 alpha, bias, relu, out, ldo, fn, stream);
  return spmm_narrow_gc<4, 16>(n, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                               alpha, bias, relu, out, ldo, fn, stream);
}

bool self_in_epilogue_supported(int64_t nnz, int32_t d, int32_t kin) {
  const int nb = q8_lane_bytes(d);
  return nnz > 0 && d <= 256 && nb >= 2 && ((kin + 63) >> 6) * nb <= 16;
}

hipError_t launch_spmm_q8(int64_t n, int64_t nnz, const int64_t* rowptr,
                          const int32_t* colidx, int mean, const float* g,
                          const int8_t* C8, int64_t ldc8, const void* C16,
                          int64_t ldc16, int32_t K, int32_t d, const float* alpha,
                          const float* bias, int relu, float* out, int64_t ldo,
                          const SpmmPlan& p, void* ws, const FusedNext* next,
                          hipStream_t stream) {
  if (n == 0) return hipSuccess;
  FusedNext none = {};
  const FusedNext& fn = next != nullptr ? *next : none;
  if (fn.kind == 3 && !self_in_epilogue_supported(nnz, d, fn.kin)) return hipErrorInvalidValue;
  if (nnz == 0 && fn.kind == 2) {
    const int64_t total = n * (int64_t)d;
    hipLaunchKernelGGL(k_sage_self_only, dim3((unsigned)((total + kBlock - 1) / kBlock)),
                       dim3(kBlock), 0, stream, n, d, g, (const _Float16*)fn.Cself,
                       fn.ldself, fn.alpha_self, bias, relu, out, ldo);
    return hipGetLastError();
  }
  if (nnz == 0 && fn.kind == 0) {
    const int64_t total = n * (int64_t)d;
    hipLaunchKernelGGL(k_spmm_empty, dim3((unsigned)((total + kBlock - 1) / kBlock)),
                       dim3(kBlock), 0, stream, n, d, bias, relu, out, ldo);
    return hipGetLastError();
  }
  if (q8_lane_bytes(d) == 1 && nnz < ((int64_t)1 << 31))
    return spmm_narrow(n, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d, alpha, bias,
                       relu, out, ldo, fn, stream);
  switch (q8_lane_bytes(d)) {
    case 1:
      return spmm_q8_nb<1>(n, nnz, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                           alpha, bias, relu, out, ldo, p, ws, fn, stream);
    case 2:
      return spmm_q8_nb<2>(n, nnz, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                           alpha, bias, relu, out, ldo, p, ws, fn, stream);
    default:
      return spmm_q8_nb<4>(n, nnz, rowptr, colidx, mean, g, C8, ldc8, C16, ldc16, K, d,
                           alpha, bias, relu, out, ldo, p, ws, fn, stream);
  }
}

// ------------------------------------------------------ source order ----
//
// The forward pass stores each node's products and scale at a slot: nodes
// listed by descending degree class (class 0 for degree <= 1, else
// floor(log2 degree)), by node id within a class.  The aggregation gathers
// a source row per edge; in a power-law graph most gathers hit a small set
// of high-degree nodes, and with them first their rows and scales share
// cache lines, so a gather hits the XCD's L2 more often.  Destination rows
// keep their order, so no input or output moves and every sum keeps its
// terms and their order.
//
// One wave per group of 64 consecutive nodes counts its nodes per class;
// an exclusive scan over (class descending, group ascending) gives each
// (class, group) its first slot; each node then takes that slot plus the
// number of lower lanes of its group in its class.

constexpr int kSlotClasses = 32;

__device__ inline int degree_class(int64_t deg) {
  return deg <= 1 ? 0 : 63 - __builtin_clzll((uint64_t)deg);
}

// counts[(31 - c) * groups + w] = nodes of group w in class c.
__global__ __launch_bounds__(kBlock) void k_slot_count(int64_t n,
                                                       const int64_t* __restrict__ rowptr,
                                                       int64_t groups,
                                                       int32_t* __restrict__ counts) {
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
  if (w >= groups) return;
  const int64_t i = w * 64 + lane;
  const int cls = i < n ? degree_class(rowptr[i + 1] - rowptr[i]) : -1;
  int mine = 0;
#pragma unroll 4
  for (int c = 0; c < kSlotClasses; ++c) {
    const int cnt = (int)__builtin_popcountll(__builtin_amdgcn_ballot_w64(cls == c));
    if (lane == c) mine = cnt;
  }
  if (lane < kSlotClasses) counts[(int64_t)(kSlotClasses - 1 - lane) * groups + w] = mine;
}

// Exclusive scan of v[0, total), in place, in three passes: block sums of
// 1024 entries, a scan of those sums by one block, then each block's scan
// plus its offset.  Entries and sums stay below 2^31 (at most n nodes).
constexpr int kScanPer = 4;
constexpr int kScanTile = kBlock * kScanPer;

__device__ inline int32_t block_exclusive_scan(int32_t v, int32_t* s_tmp, int32_t& total) {
  const int t = threadIdx.x;
  s_tmp[t] = v;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    const int32_t add = t >= off ? s_tmp[t - off] : 0;
    __syncthreads();
    s_tmp[t] += add;
    __syncthreads();
  }
  total = s_tmp[kBlock - 1];
  const int32_t incl = s_tmp[t];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(kBlock) void k_scan_sums(const int32_t* __restrict__ v,
                                                      int64_t total,
                                                      int32_t* __restrict__ sums) {
  __shared__ int32_t s_tmp[kBlock];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
  int32_t acc = 0;
#pragma unroll
  for (int u = 0; u < kScanPer; ++u) acc += base + u < total ? v[base + u] : 0;
  int32_t sum;
  block_exclusive_scan(acc, s_tmp, sum);
  if (threadIdx.x == 0) sums[blockIdx.x] = sum;
}

__global__ __launch_bounds__(kBlock) void k_scan_top(int32_t* __restrict__ sums, int64_t nb) {
  __shared__ int32_t s_tmp[kBlock];
  const int64_t per = (nb + kBlock - 1) / kBlock;
  const int64_t b0 = (int64_t)threadIdx.x * per;
  int32_t acc = 0;
  for (int64_t b = b0; b < b0 + per && b < nb; ++b) acc += sums[b];
  int32_t total;
  int32_t run = block_exclusive_scan(acc, s_tmp, total);
  for (int64_t b = b0; b < b0 + per && b < nb; ++b) {
    const int32_t x = sums[b];
    sums[b] = run;
    run += x;
  }
}

__global__ __launch_bounds__(kBlock) void k_scan_apply(int32_t* __restrict__ v, int64_t total,
                                                       const int32_t* __restrict__ sums) {
  __shared__ int32_t s_tmp[kBlock];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
  int32_t x[kScanPer];
  int32_t acc = 0;
#pragma unroll
  for (int u = 0; u < kScanPer; ++u) {
    x[u] = base + u < total ? v[base + u] : 0;
    acc += x[u];
  }
  int32_t unused;
  int32_t run = sums[blockIdx.x] + block_exclusive_scan(acc, s_tmp, unused);
#pragma unroll
  for (int u = 0; u < kScanPer; ++u) {
    if (base + u < total) v[base + u] = run;
    run += x[u];
  }
}

__global__ __launch_bounds__(kBlock) void k_slot_scatter(int64_t n,
                                                         const int64_t* __restrict__ rowptr,
                                                         int64_t groups,
                                                         const int32_t* __restrict__ first,
                                                         int32_t* __restrict__ slot) {
  const int lane = threadIdx.x & 63;
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + wave_index_in_block();
  if (w >= groups) return;
  const int64_t i = w * 64 + lane;
  const int cls = i < n ? degree_class(rowptr[i + 1] - rowptr[i]) : -1;
  const uint64_t below = (1ull << lane) - 1;
  int rank = 0;
#pragma unroll 4
  for (int c = 0; c < kSlotClasses; ++c) {
    const uint64_t m = __builtin_amdgcn_ballot_w64(cls == c);
    if (cls == c) rank = (int)__builtin_popcountll(m & below);
  }
  if (i < n) slot[i] = first[(int64_t)(kSlotClasses - 1 - cls) * groups + w] + rank;
}

__global__ __launch_bounds__(kBlock) void k_colslot(int64_t nnz,
                                                    const int32_t* __restrict__ colidx,
                                                    const int32_t* __restrict__ slot,
                                                    int32_t* __restrict__ colslot) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < nnz; e += stride)
    colslot[e] = slot[colidx[e]];
}

SlotPlan source_slots_plan(int64_t n) {
  SlotPlan p;
  p.groups = (n + 63) / 64;
  p.total = p.groups * kSlotClasses;
  p.blocks = (p.total + kScanTile - 1) / kScanTile;
  auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
  p.off_sums = up((size_t)p.total * 4);
  p.bytes = p.off_sums + up((size_t)(p.blocks > 0 ? p.blocks : 1) * 4);
  return p;
}

hipError_t launch_source_slots(int64_t n, int64_t nnz, const int64_t* rowptr,
                               const int32_t* colidx, int32_t* slot, int32_t* colslot,
                               void* ws, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const SlotPlan p = source_slots_plan(n);
  int32_t* counts = (int32_t*)ws;
  int32_t* sums = (int32_t*)((char*)ws + p.off_sums);
  const dim3 wgrid((unsigned)((p.groups + kWavesPerBlock - 1) / kWavesPerBlock));
  hipLaunchKernelGGL(k_slot_count, wgrid, dim3(kBlock), 0, stream, n, rowptr, p.groups,
                     counts);
  hipLaunchKernelGGL(k_scan_sums, dim3((unsigned)p.blocks), dim3(kBlock), 0, stream, counts,
                     p.total, sums);
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, stream, sums, p.blocks);
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)p.blocks), dim3(kBlock), 0, stream, counts,
                     p.total, sums);
  hipLaunchKernelGGL(k_slot_scatter, wgrid, dim3(kBlock), 0, stream, n, rowptr, p.groups,
                     counts, slot);
  if (nnz > 0)
    hipLaunchKernelGGL(k_colslot, dim3(grid_cap((nnz + kBlock - 1) / kBlock, 8192)),
                       dim3(kBlock), 0, stream, nnz, colidx, slot, colslot);
  return hipGetLastError();
}

bool bgemm_mfma_supported(int32_t N, int32_t K) { return N >= 1 && N <= 256 && K >= 1; }

template <int NT>
static void launch_mfma_nt(dim3 grid, size_t lds, hipStream_t stream, const uint64_t* F,
                           int64_t M, int64_t ldf, const uint64_t* B, int32_t N,
                           int64_t ldb, int32_t K, void* C, IType ct, int64_t ldc,
                           int32_t groups, int32_t kc_max) {
  switch (ct) {
    case IType::F16:
      hipLaunchKernelGGL((k_bgemm_mfma<NT, _Float16>), grid, dim3(kBlock), lds, stream, F,
                         M, ldf, B, N, ldb, K, (_Float16*)C, ldc, groups, kc_max);
      break;
    case IType::I16:
      hipLaunchKernelGGL((k_bgemm_mfma<NT, int16_t>), grid, dim3(kBlock), lds, stream, F,
                         M, ldf, B, N, ldb, K, (int16_t*)C, ldc, groups, kc_max);
      break;
    default:
      hipLaunchKernelGGL((k_bgemm_mfma<NT, int32_t>), grid, dim3(kBlock), lds, stream, F,
                         M, ldf, B, N, ldb, K, (int32_t*)C, ldc, groups, kc_max);
      break;
  }
}

hipError_t launch_bgemm_mfma(const uint64_t* F, int64_t M, int64_t ldf, const uint64_t* B,
                             int32_t N, int64_t ldb, int32_t K, void* C, IType ct,
                             int64_t ldc, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int kw = (K + 63) / 64;
  const int tiles = (N + 15) / 16;
  // Column tiles per block: a power of two <= 8, halved while the block's
  // expanded weights (1 KB per tile and word) would not stay resident.
  int NT = 1;
  while (NT < tiles && NT < 8) NT *= 2;
  while (NT > 1 && (size_t)kw * NT * 1024 > (size_t)kMfmaLdsBytes) NT /= 2;
  const int groups = (tiles + NT - 1) / NT;
  const int kc_max = std::min(kw, kMfmaLdsBytes / (NT * 1024));
  const size_t lds = (size_t)kc_max * NT * 1024;
  const int64_t row_blocks = (M + kWavesPerBlock * 32 - 1) / (kWavesPerBlock * 32);
  const int64_t cap = 4096 - 4096 % groups;
  const dim3 grid((unsigned)std::min<int64_t>(row_blocks * groups, cap));
  switch (NT) {
    case 1: launch_mfma_nt<1>(grid, lds, stream, F, M, ldf, B, N, ldb, K, C, ct, ldc, groups, kc_max); break;
    case 2: launch_mfma_nt<2>(grid, lds, stream, F, M, ldf, B, N, ldb, K, C, ct, ldc, groups, kc_max); break;
    case 4: launch_mfma_nt<4>(grid, lds, stream, F, M, ldf, B, N, ldb, K, C, ct, ldc, groups, kc_max); break;
    default: launch_mfma_nt<8>(grid, lds, stream, F, M, ldf, B, N, ldb, K, C, ct, ldc, groups, kc_max); break;
  }
  return hipGetLastError();
}

}  // namespace bigcn
