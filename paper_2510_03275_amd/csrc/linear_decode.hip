// Decode path of sdq_linear (m <= 16 activation rows), two launches each.
//
// One activation row (addition-only):
//   expand   x_tilde_b = x_b E for every block b, E = Had D^T (B x M, fp32; D is
//            the Resample back to B).  A workgroup owns 64 output samples of
//            one block (one wave per quarter of t, E held in registers) and
//            all activation rows.  The workgroups also zero y when the GEMV
//            will split K.
//   gemv     y[i, r] = s_r * sum_j C[r, j] x_tilde[i, j] with additions only: a
//            workgroup owns one K segment and four 64-row panels (one per
//            wave, lane = weight row).  It first issues the loads of its
//            16-byte code chunks (coalesced 1 KB per wave), then builds the
//            segment's lookup tables of the 16 signed partial sums of every
//            4-bit group of codes (4 binary codes or 2 ternary codes), and each
//            lane adds one table entry per 4 bits.
// Two to sixteen rows (integer matrix cores):
//   expand   the same x_tilde (for fp16 and bf16 x on the matrix cores, with
//            E as an fp16 pair hi + lo), quantised per (row, block) to
//            24-bit fixed point and written as three signed-byte planes;
//   gemv     codes expanded to int8 {-1, 0, +1} by a byte permute and
//            contracted against the planes with v_mfma_i32_16x16x64_i8 (exact
//            int32 sums), dequantised per block.  The cost barely grows with
//            the row count, where the table GEMV's grows linearly.
// When K is split over workgroups, each adds its scaled partial sums into y
// with fp32 atomics (y zeroed by the expansion, or holding the values to
// accumulate onto), so results can differ between runs in the last bits; an
// unsplit layer stores.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <hip/hip_bf16.h>

#include <cstdio>
#include <cstdlib>
#include <algorithm>
#include <string>

#include "sdq_internal.h"

namespace sdq {
namespace {

constexpr int kExpThreads = 256;
constexpr int kMaxDecodeRows = 16;  // activation rows of the decode path
constexpr int kGemvWaves = 4;
constexpr int kGroupsPerChunk = 32; // 128 bits / 4
constexpr int64_t kExpRowPairs = 1024; // one-row expansion: two blocks per workgroup from here
constexpr int64_t kPlanePairs = 768;   // plane expansion: two blocks per workgroup from here

// A 16-byte load of packed codes, marked non-temporal: each code byte is read
// once per call, and the streaming hint keeps the code stream from evicting
// the expansion tables and x_tilde from L2 (measured on MI355X: the 70B stack
// at m = 1 9.94 -> 9.47 ms per token, at m = 8 16.08 -> 15.55 ms).
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* dec_lds_ptr;
typedef __attribute__((address_space(1))) const void* dec_gbl_ptr;
constexpr int kWaitVm0 = 7 << 4;   // s_waitcnt vmcnt(0) lgkmcnt(0), expcnt not waited on

__device__ inline uint4 load_code_chunk(const uint4* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ inline float load_x(const void* x, sdq_dtype xt, int64_t idx) {
  if (xt == SDQ_F16) return __half2float(static_cast<const __half*>(x)[idx]);
  if (xt == SDQ_BF16) return __bfloat162float(static_cast<const __hip_bfloat16*>(x)[idx]);
  return static_cast<const float*>(x)[idx];
}

// Zero the outputs of a set of linears (m rows each), grid-stride over the
// launch's workgroups: a side duty of the expansion when the GEMV that follows
// adds its split-K partials into y.
__device__ inline void zero_outputs(const LinearSet& z, int m, int64_t wg, int64_t n_wg, int tid) {
  for (int j = 0; j < z.count; ++j) {
    const int64_t cnt = static_cast<int64_t>(m) * z.n[j];
    float* p = z.y[j];
    for (int64_t i = wg * kExpThreads + tid; i < cnt; i += n_wg * kExpThreads) p[i] = 0.0f;
  }
}

// The linear of a set that unit u of a launch belongs to (first[] holds the
// prefix sums of the units per linear); uniform over the workgroup.
__device__ inline int linear_of(const LinearSet& S, int64_t u) {
  int j = 0;
#pragma unroll
  for (int i = 1; i < kMaxGroup; ++i)
    if (i < S.count && u >= S.first[i]) j = i;
  return j;
}

// One workgroup: 64 output samples of one block, all m rows.  Wave w keeps
// the quarter t in [w B/4, (w+1) B/4) of the 64 columns of E in registers
// (the grouped table layout makes each of its loads 1 KB contiguous); the
// activation block is staged in LDS as fp32, and the four partial dots of
// each output meet in LDS.
template <int B>
__global__ __launch_bounds__(kExpThreads) void expand_decode_kernel(
    const void* __restrict__ x, sdq_dtype xt, int m, int64_t k, int m_up, int m_pad,
    int64_t k_up, int64_t k_up_pad, const float4* __restrict__ edec, float* __restrict__ xt_out,
    LinearSet zero) {
  constexpr int TQ = B / 4;                 // t values per wave
  __shared__ float xs[kMaxDecodeRows][B];
  __shared__ float red[4][kMaxDecodeRows][64];
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int w = tid / 64;
  const int o = blockIdx.x * 64 + lane;     // < m_pad: the table is zero there
  const int64_t b = blockIdx.y;
  float4 e[TQ / 4];
  const float4* ep = edec + static_cast<int64_t>(w * (TQ / 4)) * m_pad + o;
#pragma unroll
  for (int q = 0; q < TQ / 4; ++q) e[q] = ep[static_cast<int64_t>(q) * m_pad];
  for (int idx = tid; idx < m * B; idx += kExpThreads) {
    const int i = idx / B, t = idx % B;
    xs[i][t] = load_x(x, xt, static_cast<int64_t>(i) * k + b * B + t);
  }
  // Side duties: zero y for a split-K GEMV, zero x_tilde's padding.
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t n_wg = static_cast<int64_t>(gridDim.x) * gridDim.y;
  zero_outputs(zero, m, wg, n_wg, tid);
  if (wg == 0) {
    const int64_t pad = k_up_pad - k_up;
    for (int64_t i = tid; i < m * pad; i += kExpThreads)
      xt_out[(i / pad) * k_up_pad + k_up + (i % pad)] = 0.0f;
  }
  __syncthreads();
  for (int i = 0; i < m; ++i) {
    const float4* xr = reinterpret_cast<const float4*>(&xs[i][w * TQ]);
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
    for (int q = 0; q < TQ / 4; ++q) {
      const float4 v = xr[q];
      a0 += e[q].x * v.x;
      a1 += e[q].y * v.y;
      a2 += e[q].z * v.z;
      a3 += e[q].w * v.w;
    }
    red[w][i][lane] = (a0 + a1) + (a2 + a3);
  }
  __syncthreads();
  for (int idx = tid; idx < m * 64; idx += kExpThreads) {
    const int i = idx / 64, l = idx % 64;
    const int oo = blockIdx.x * 64 + l;
    if (oo < m_up)
      xt_out[static_cast<int64_t>(i) * k_up_pad + b * m_up + oo] =
          (red[0][i][l] + red[1][i][l]) + (red[2][i][l] + red[3][i][l]);
  }
}

// One activation row: one workgroup per 64 output samples and NBW (1 or 2)
// consecutive blocks.  The 64 columns of E are loaded once into registers
// (wave w: t in its quarter, as above) and serve every block of the
// workgroup, and the x of all its blocks is staged in LDS by one round of
// loads issued together, so E crosses the caches once per NBW blocks instead
// of once per block.  Same sums in the same order as expand_decode_kernel.
template <int B, int NBW>
__global__ __launch_bounds__(kExpThreads) void expand_decode_row_kernel(
    const void* __restrict__ x, sdq_dtype xt, int nb, int m_up, int m_pad, int64_t k_up, int64_t k_up_pad,
    const float4* __restrict__ edec, float* __restrict__ xt_out, LinearSet zero) {
  constexpr int TQ = B / 4;                 // t values per wave
  constexpr int XPT = (NBW * B + kExpThreads - 1) / kExpThreads;  // x values staged per thread
  __shared__ float xs[NBW][B];
  __shared__ float red[4][NBW][64];
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int w = tid / 64;
  const int o = blockIdx.x * 64 + lane;     // < m_pad: the table is zero there
  const int b0 = blockIdx.y * NBW;
  const int nbl = min(NBW, nb - b0);
  float4 e[TQ / 4];
  const float4* ep = edec + static_cast<int64_t>(w * (TQ / 4)) * m_pad + o;
#pragma unroll
  for (int q = 0; q < TQ / 4; ++q) e[q] = ep[static_cast<int64_t>(q) * m_pad];
  float xv[XPT];
#pragma unroll
  for (int j = 0; j < XPT; ++j) {
    const int idx = tid + kExpThreads * j;
    xv[j] = idx < NBW * B && idx / B < nbl ? load_x(x, xt, static_cast<int64_t>(b0) * B + idx) : 0.0f;
  }
#pragma unroll
  for (int j = 0; j < XPT; ++j) {
    const int idx = tid + kExpThreads * j;
    if (idx < NBW * B) xs[idx / B][idx % B] = xv[j];
  }
  // Side duties: zero y for a split-K GEMV, zero x_tilde's padding.
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t n_wg = static_cast<int64_t>(gridDim.x) * gridDim.y;
  zero_outputs(zero, 1, wg, n_wg, tid);
  if (wg == 0)
    for (int64_t i = k_up + tid; i < k_up_pad; i += kExpThreads) xt_out[i] = 0.0f;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    if (j >= nbl) break;
    const float4* xr = reinterpret_cast<const float4*>(&xs[j][w * TQ]);
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
    for (int q = 0; q < TQ / 4; ++q) {
      const float4 v = xr[q];
      a0 += e[q].x * v.x;
      a1 += e[q].y * v.y;
      a2 += e[q].z * v.z;
      a3 += e[q].w * v.w;
    }
    red[w][j][lane] = (a0 + a1) + (a2 + a3);
  }
  __syncthreads();
  for (int idx = tid; idx < nbl * 64; idx += kExpThreads) {
    const int j = idx / 64, l = idx % 64;
    const int oo = blockIdx.x * 64 + l;
    if (oo < m_up)
      xt_out[static_cast<int64_t>(b0 + j) * m_up + oo] =
          (red[0][j][l] + red[1][j][l]) + (red[2][j][l] + red[3][j][l]);
  }
}

// ---------------------------------------------------------------------------
// Integer-MFMA decode: x_tilde as 24-bit fixed point in three signed-byte
// planes, codes expanded to int8 (+-1 binary, 64 x {-1, 0, +1} ternary),
// exact int32 accumulation (|sum| <= 128 * 64 * M per block).
//
// Per (activation row i, block b) the scale is S = max_t |x_b[t]| * e1max / Q
// with e1max >= max_m sum_t |E[t][m]|, so |x_tilde_b| <= Q * S and the rounded
// value q = rint(x_tilde / S) splits into bytes h, m, l in [-128, 127] with
// q = 65536 h + 256 m + l.  Every workgroup of a block computes the same S
// from the same staged block (a max is order independent).
//
// k-steps of 64 codes (v_mfma_i32_16x16x64_i8: lane l holds row l % 16 and
// the 16 bytes of k-group kg = l / 16).  The planes are laid out per block:
// block b owns cpb chunk slots, slot j holding the samples of code chunk
// floor(b M / chunk) + j that belong to block b and zeros elsewhere, so a
// block that starts or ends inside a chunk (M not a multiple of the chunk)
// shares that chunk's codes with its neighbour but not its planes, and every
// k-step sums one block only; cpb is the most chunks any block touches.
// Inside a chunk the codes map to (step, kg, dword di, byte beta) as
// code_bytes produces them from the chunk's word kg:
//   ternary  one step per chunk,  code 16 kg + di + 4 beta      (fields di + 4 beta)
//   binary   two steps s per chunk, code 32 kg + 4 s + di + 8 beta  (bits 4 s + di + 8 beta)
// A = planes: row p = 4 a + t (activation row a of the plane group, plane t:
// h, m, l, zero), stored per step and plane group as 64 lanes x 16 bytes.
constexpr float kQ = 8257536.0f;    // 2^23 - 2^17: leaves |h| <= 126

// B-operand bytes of four codes of a chunk word: byte beta holds code field
// (or bit) d of the word's byte beta.  Ternary fields move to the top two bits
// of their byte, which as a signed byte is 64 x code (0b01 -> 64, 0b11 -> -64,
// 0b00 -> 0): a shift and a mask, with the factor 64 (kCodeScale) divided out of
// the block's sums, exactly, with the plane scale.  Binary bits 0 / 1 map to
// -1 / +1 through a byte permute.
template <int LEVELS>
__device__ inline int code_bytes(uint32_t wv, int d) {
  if constexpr (LEVELS == 2)
    return static_cast<int>(__builtin_amdgcn_perm(0u, 0x000001FFu, (wv >> d) & 0x01010101u));
  else
    return static_cast<int>((wv << (6 - 2 * d)) & 0xC0C0C0C0u);
}
template <int LEVELS>
constexpr float kCodeScale = LEVELS == 2 ? 1.0f : 64.0f;

template <int LEVELS>
__device__ inline int chunk_code(int s, int kg, int di, int beta) {
  return LEVELS == 2 ? 32 * kg + 4 * s + di + 8 * beta : 16 * kg + di + 4 * beta;
}

__device__ inline uint32_t plane_byte(int q, int t) {
  const int l = ((q + 128) & 255) - 128;
  const int q1 = (q - l) >> 8;
  const int mm = ((q1 + 128) & 255) - 128;
  const int h = (q1 - mm) >> 8;
  const int v = t == 0 ? h : (t == 1 ? mm : (t == 2 ? l : 0));
  return static_cast<uint32_t>(v) & 255u;
}

// Max over the 64 lanes of a wave of non-negative floats (compared as their
// bit patterns, which order them alike): DPP steps within each row of 16
// lanes, then the row broadcasts carry rows 0-2 into row 3; read from lane 63.
__device__ inline float wave_max_nonneg(float v) {
  int x = __float_as_int(v);
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));    // quad_perm [1, 0, 3, 2]
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));    // quad_perm [2, 3, 0, 1]
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));   // row_half_mirror
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));   // row_mirror
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false));   // row_bcast:15 -> rows 1, 3
  x = max(x, __builtin_amdgcn_update_dpp(x, x, 0x143, 0xC, 0xF, false));   // row_bcast:31 -> rows 2, 3
  return __int_as_float(__builtin_amdgcn_readlane(x, 63));
}

// The plane words of one workgroup's 64 code positions (2-bit fields):
// chunk slot `slot`, and (binary) half `half` of the chunk, from the
// quantised samples qv[row][position] of all m rows (rows >= m and plane 3
// zero); 256 * npg dwords, every thread of the workgroup taking a share.
template <int LEVELS>
__device__ inline void store_planes(const int (*qv)[64], int m, int npg, int64_t slot, int half,
                                    uint32_t* __restrict__ planes) {
  for (int idx = threadIdx.x; idx < 256 * npg; idx += kExpThreads) {
    const int di = idx % 4;
    const int p = (idx / 4) % 16;
    int s, kg, pg;
    if (LEVELS == 2) {          // kg in {2 half, 2 half + 1}, both steps of the chunk
      kg = 2 * half + (idx / 64) % 2;
      pg = (idx / 128) % npg;
      s = idx / (128 * npg);
    } else {                    // all four kg, the chunk's one step
      kg = (idx / 64) % 4;
      pg = idx / 256;
      s = 0;
    }
    const int a = pg * 4 + p / 4;
    const int t = p % 4;
    uint32_t word = 0;
    if (a < m && t < 3) {
#pragma unroll
      for (int beta = 0; beta < 4; ++beta)
        word |= plane_byte(qv[a][chunk_code<LEVELS>(s, kg, di, beta) - 64 * half], t) << (8 * beta);
    }
    const int64_t step = LEVELS == 2 ? 2 * slot + s : slot;
    planes[((step * npg + pg) * 64 + kg * 16 + p) * 4 + di] = word;
  }
}

// One activation row: the planes h, m, l of the workgroup's 64 code
// positions in the compact layout of that case, 12 groups of 16 bytes per
// k-step (k-group kg, plane t at (kg * 3 + t) * 16 bytes) -- the A-operand
// words of lanes 16 kg + t; the other lanes' rows are zero and not stored.
// Lanes idx < 48 of one wave store a dword each.
template <int LEVELS>
__device__ inline void store_planes_m1(const int* qv, int64_t slot, int half, int idx,
                                       uint32_t* __restrict__ planes) {
  if (idx >= 48) return;
  const int di = idx % 4;
  const int t = (idx / 4) % 3;
  int s, kg;
  if (LEVELS == 2) {
    kg = 2 * half + (idx / 12) % 2;
    s = idx / 24;
  } else {
    kg = idx / 12;
    s = 0;
  }
  uint32_t word = 0;
#pragma unroll
  for (int beta = 0; beta < 4; ++beta)
    word |= plane_byte(qv[chunk_code<LEVELS>(s, kg, di, beta) - 64 * half], t) << (8 * beta);
  const int64_t step = LEVELS == 2 ? 2 * slot + s : slot;
  planes[((step * 12) + kg * 3 + t) * 4 + di] = word;
}

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

// Matrix-core front end of the plane expansions for fp16 and bf16
// activations: the quantised x_tilde of code positions g0 + [0, 64) of blocks
// b0 .. b0 + nbl - 1 (nbl <= NB) for all rows, into qv[j][row][position] (zero
// outside the block), and (when write_sx) the blocks' plane scales.  The
// blocks share the columns of E: with M a multiple of the code chunk, code
// position p of slot u is sample 64 u + p of every block, so E is loaded once
// per workgroup whatever NB.  Wave w takes positions 16 w + [0, 16): x_b (rows
// as the A operand, zero past m) times the columns of E as the fp16 pair hi +
// lo of the transposed tables (the B operand), 2 B / 32
// v_mfma_f32_16x16x32_f16 per block with fp32 accumulation.  bf16 x is scaled
// per (row, block) by a power of two that brings its max into [2^14, 2^15), so
// it converts to fp16 exactly (values below 2^-24 of the max round); the scale
// cancels in the quantisation, whose bound max |x_b| * e1max is the fp32
// path's.  E hi + lo carries ~22 bits, against 24 for the fixed point.
template <int B, bool BF16, int NB>
__device__ inline void planes_qv_mfma(const uint16_t* __restrict__ x, int m, int k32, int64_t b0, int nbl,
                                      int64_t g0, int m_up, int64_t nb, bool write_sx,
                                      const uint16_t* __restrict__ et_hi, const uint16_t* __restrict__ et_lo,
                                      float e1max, float* __restrict__ sx, int (*qv)[kMaxDecodeRows][64]) {
  constexpr int S = B / 32;                  // k-steps of 32 samples of t
  const int lane = threadIdx.x % 64;
  const int w = threadIdx.x / 64;
  const int r = lane % 16, grp = lane / 16;  // operand row / column, k group
  const int pos = 16 * w + r;                // this lane's B column: code position
  const int o = static_cast<int>(g0 + pos - b0 * m_up);
  const bool in_block = o >= 0 && o < m_up;
  // Loads from clamped (in-bounds) addresses, zeroed by selects.
  const uint4* __restrict__ hp = reinterpret_cast<const uint4*>(et_hi + static_cast<int64_t>(in_block ? o : 0) * B) + grp;
  const uint4* __restrict__ lp = reinterpret_cast<const uint4*>(et_lo + static_cast<int64_t>(in_block ? o : 0) * B) + grp;
  uint4 xq[NB][S], eh[S], el[S];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t bj = b0 + min(j, nbl - 1);
    const uint4* __restrict__ xp =
        reinterpret_cast<const uint4*>(x + static_cast<int64_t>(min(r, m - 1)) * k32 + bj * B) + grp;
#pragma unroll
    for (int st = 0; st < S; ++st) xq[j][st] = xp[4 * st];
  }
#pragma unroll
  for (int st = 0; st < S; ++st) eh[st] = hp[4 * st];
#pragma unroll
  for (int st = 0; st < S; ++st) el[st] = lp[4 * st];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    if (j >= nbl) break;
    // max |x| of row r over the lane's 8 S samples, then over the four k groups
    float mx = 0.0f;
#pragma unroll
    for (int st = 0; st < S; ++st) {
      const uint32_t wv[4] = {xq[j][st].x, xq[j][st].y, xq[j][st].z, xq[j][st].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float lo = BF16 ? __uint_as_float(wv[q] << 16)
                              : __half2float(__ushort_as_half(static_cast<unsigned short>(wv[q])));
        const float hi = BF16 ? __uint_as_float(wv[q] & 0xFFFF0000u)
                              : __half2float(__ushort_as_half(static_cast<unsigned short>(wv[q] >> 16)));
        mx = fmaxf(mx, fmaxf(fabsf(lo), fabsf(hi)));
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (r >= m) mx = 0.0f;
    int ex = 0;
    (void)frexpf(mx, &ex);                     // mx < 2^ex
    const int sh = mx > 0.0f ? 15 - ex : 0;    // bf16 scale 2^sh
    float4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int st = 0; st < S; ++st) {
      half8_t a;
      if constexpr (BF16) {
        const uint32_t wv[4] = {xq[j][st].x, xq[j][st].y, xq[j][st].z, xq[j][st].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          a[2 * q] = static_cast<_Float16>(ldexpf(__uint_as_float(wv[q] << 16), sh));
          a[2 * q + 1] = static_cast<_Float16>(ldexpf(__uint_as_float(wv[q] & 0xFFFF0000u), sh));
        }
      } else {
        a = *reinterpret_cast<const half8_t*>(&xq[j][st]);
      }
      if (r >= m) a = half8_t{0, 0, 0, 0, 0, 0, 0, 0};
      half8_t h = *reinterpret_cast<const half8_t*>(&eh[st]);
      half8_t l = *reinterpret_cast<const half8_t*>(&el[st]);
      if (!in_block) {
        h = half8_t{0, 0, 0, 0, 0, 0, 0, 0};
        l = h;
      }
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, h, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, l, acc, 0, 0, 0);
    }
    // Output v of this lane: row a = 4 grp + v, position pos.  The row's max
    // sits in lane a (lane a holds row a % 16 = a).
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int a = 4 * grp + v;
      const float mxa = __shfl(mx, a);
      const float bound = mxa * e1max;
      int q = 0;
      if (bound > 0.0f && in_block) {
        int exa = 0;
        (void)frexpf(mxa, &exa);
        const float sc = BF16 ? ldexpf(bound, 15 - exa) : bound;   // the bound in acc's scale
        q = __float2int_rn(acc[v] * (kQ / sc));
      }
      qv[j][a][pos] = q;
    }
    if (write_sx && w == 0 && grp == 0 && r < m) sx[static_cast<int64_t>(r) * nb + b0 + j] = mx * e1max / kQ;
  }
}

// One workgroup: one 64-code segment u of block b's chunk slots (code
// positions floor(b M / chunk) * chunk + 64 u + [0, 64)), all m rows; the
// samples of block b among them by the fp32 expansion, the rest zero; then
// quantised and written as planes (256 * npg dwords per workgroup; one row:
// 48 dwords in the compact layout).  NB = 2 (one activation row, M a multiple
// of the chunk): blocks b and b + 1 take the places of two rows, sharing the
// workgroup's columns of E.
template <int B, int LEVELS, int NB>
__global__ __launch_bounds__(kExpThreads) void expand_planes_kernel(
    const void* __restrict__ x, sdq_dtype xt, int m, int npg, int64_t k, int64_t nb, int m_up,
    int m_pad, int cpb, const float4* __restrict__ edec, float e1max, uint32_t* __restrict__ planes,
    float* __restrict__ sx, LinearSet zero) {
  constexpr int TQ = B / 4;
  __shared__ float xs[kMaxDecodeRows][B];
  __shared__ float red[4][kMaxDecodeRows][64];
  __shared__ int qv[kMaxDecodeRows][64];
  __shared__ float xmax[kMaxDecodeRows];
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int w = tid / 64;
  constexpr int kCpc = LEVELS == 2 ? 128 : 64;             // codes per chunk
  static_assert(NB == 1 || NB == 2, "one or two blocks per workgroup");
  const int64_t b = static_cast<int64_t>(blockIdx.y) * NB;
  // rows of the workgroup: the m activation rows, or (NB = 2) the blocks
  const int R = NB == 2 ? static_cast<int>(min<int64_t>(2, nb - b)) : m;
  const int64_t c_first = b * m_up / kCpc;                  // block b's first code chunk
  const int64_t g0 = c_first * kCpc + static_cast<int64_t>(blockIdx.x) * 64;
  const int o = static_cast<int>(g0 + lane - b * m_up);    // this lane's sample within block b
  const bool in_block = o >= 0 && o < m_up;
  // The activation block goes to LDS with every load issued before any
  // store (converted afterwards: a conversion next to its load waits for it,
  // one global round trip per element), and before the E columns, so that
  // the stores and the max below wait for x alone.
  constexpr int XPT = kMaxDecodeRows * B / kExpThreads;   // elements per thread, at most
  const int mb = R * B;
  uint32_t xr[XPT];
  // row stride: k (activation rows), or B (consecutive blocks of row 0)
  const int k32 = NB == 2 ? B : static_cast<int>(k);   // m k < 2^31 on the decode path
  if (xt == SDQ_F32) {
    const uint32_t* __restrict__ xp = static_cast<const uint32_t*>(x) + b * B;
#pragma unroll
    for (int r = 0; r < XPT; ++r) {
      if (kExpThreads * r >= mb) break;
      const int idx = tid + kExpThreads * r;
      xr[r] = idx < mb ? xp[(idx / B) * k32 + idx % B] : 0u;
    }
  } else {
    const uint16_t* __restrict__ xp = static_cast<const uint16_t*>(x) + b * B;
#pragma unroll
    for (int r = 0; r < XPT; ++r) {
      if (kExpThreads * r >= mb) break;
      const int idx = tid + kExpThreads * r;
      xr[r] = idx < mb ? xp[(idx / B) * k32 + idx % B] : 0u;
    }
  }
  float4 e[TQ / 4];
  const float4* ep = edec + static_cast<int64_t>(w * (TQ / 4)) * m_pad + (in_block ? o : 0);
#pragma unroll
  for (int q = 0; q < TQ / 4; ++q) e[q] = ep[static_cast<int64_t>(q) * m_pad];
#pragma unroll
  for (int r = 0; r < XPT; ++r) {
    if (kExpThreads * r >= mb) break;
    const int idx = tid + kExpThreads * r;
    if (idx < mb) {
      const float v = xt == SDQ_F32    ? __uint_as_float(xr[r])
                      : xt == SDQ_BF16 ? __uint_as_float(xr[r] << 16)
                                       : __half2float(__ushort_as_half(static_cast<unsigned short>(xr[r])));
      xs[idx / B][idx % B] = v;
    }
  }
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t n_wg = static_cast<int64_t>(gridDim.x) * gridDim.y;
  zero_outputs(zero, m, wg, n_wg, tid);
  __syncthreads();
  // max |x_b| per row: wave w handles rows w, w + 4, ...
  for (int i = w; i < R; i += 4) {
    float mx = 0.0f;
    for (int t = lane; t < B; t += 64) mx = fmaxf(mx, fabsf(xs[i][t]));
    mx = wave_max_nonneg(mx);
    if (lane == 0) xmax[i] = mx;
  }
  for (int i = 0; i < R; ++i) {
    const float4* xr = reinterpret_cast<const float4*>(&xs[i][w * TQ]);
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
    for (int q = 0; q < TQ / 4; ++q) {
      const float4 v = xr[q];
      a0 += e[q].x * v.x;
      a1 += e[q].y * v.y;
      a2 += e[q].z * v.z;
      a3 += e[q].w * v.w;
    }
    red[w][i][lane] = (a0 + a1) + (a2 + a3);
  }
  __syncthreads();
  const int64_t u = static_cast<int64_t>(blockIdx.x) / (kCpc / 64);
  const int half = static_cast<int>(blockIdx.x % (kCpc / 64));
  if (m == 1) {
    // wave i finishes row (block) i alone: sum, quantise, compact plane words
    if (w < R) {
      const int i = w;
      const float val = (red[0][i][lane] + red[1][i][lane]) + (red[2][i][lane] + red[3][i][lane]);
      const float bound = xmax[i] * e1max;
      qv[i][lane] = bound > 0.0f && in_block ? __float2int_rn(val * (kQ / bound)) : 0;
      if (blockIdx.x == 0 && lane == 0) sx[NB == 2 ? b + i : b] = bound / kQ;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      store_planes_m1<LEVELS>(qv[i], (b + i) * cpb + u, half, lane, planes);
    }
    return;
  }
  for (int idx = tid; idx < R * 64; idx += kExpThreads) {
    const int i = idx / 64, l = idx % 64;
    const float val = (red[0][i][l] + red[1][i][l]) + (red[2][i][l] + red[3][i][l]);
    const float bound = xmax[i] * e1max;
    const int ol = static_cast<int>(g0 + l - b * m_up);   // (NB = 2: the same for both blocks)
    qv[i][l] = bound > 0.0f && ol >= 0 && ol < m_up ? __float2int_rn(val * (kQ / bound)) : 0;
    if (blockIdx.x == 0 && l == 0) sx[NB == 2 ? b + i : static_cast<int64_t>(i) * nb + b] = bound / kQ;
  }
  __syncthreads();
  store_planes<LEVELS>(qv, m, npg, b * cpb + u, half, planes);
}

// Base-3 codes on the integer-MFMA path (read as stored, no unpack pass).
// A base-3 chunk holds 80 codes of a row, five per byte (first code the most
// significant digit).  The k order of the contraction follows the digits:
// block b owns cpb3 chunk slots (rounded up to whole groups of four), slot j
// starting at chunk floor(b M / 80) + j; each group of four slots gives five
// 64-code k-steps: one per slot with digits 0-3 of its 16 bytes (k-group kg,
// dword di, byte beta <-> digit di of byte 4 kg + beta), and one with digit 4
// of all four slots (dword di <-> slot 4 G + di, byte beta <-> byte
// 4 kg + beta).  The planes are laid out per (block, step, plane group) as for
// the 2-bit codes.
constexpr int kB3Group = 4;    // slots per group of steps
constexpr int kB3Steps = 5;    // k-steps per group

// The plane bytes of one workgroup's 64 base-3 code positions g0 + [0, 64)
// of block b (whose first chunk is c_first) in the digit order, from
// qv[row][position]: entry idx = position (fastest), MFMA row p, plane group.
__device__ inline void store_planes_b3(const int (*qv)[64], int m, int npg, int64_t b, int64_t g0, int64_t c_first,
                                       int steps3, uint8_t* __restrict__ planes) {
  for (int idx = threadIdx.x; idx < 64 * 16 * npg; idx += kExpThreads) {
    const int l = idx % 64, p = (idx / 64) % 16, pg = idx / 1024;
    const int64_t g = g0 + l;
    const int j = static_cast<int>(g / kBase3PerChunk - c_first);
    const int pos = static_cast<int>(g % kBase3PerChunk);
    const int byte = pos / 5, digit = pos % 5;
    const int kg = byte / 4, beta = byte % 4;
    const int step = (j / kB3Group) * kB3Steps + (digit < 4 ? j % kB3Group : 4);
    const int di = digit < 4 ? digit : j % kB3Group;
    const int a = pg * 4 + p / 4, t = p % 4;
    const uint32_t val = a < m && t < 3 ? plane_byte(qv[a][l], t) : 0u;
    planes[((((b * steps3 + step) * npg + pg) * 64 + kg * 16 + p) * 16) + 4 * di + beta] = static_cast<uint8_t>(val);
  }
}

// One workgroup: 64 consecutive code positions of block b's slots (segment u
// of the block's 5 * groups segments), all m rows: the same fp32 expansion
// and 24-bit quantisation as expand_planes_kernel, then every plane byte of
// those codes (all 16 MFMA rows of each plane group, zero where no activation
// row or plane) written to its place in the digit order.
template <int B>
__global__ __launch_bounds__(kExpThreads) void expand_planes_b3_kernel(
    const void* __restrict__ x, sdq_dtype xt, int m, int npg, int64_t k, int64_t nb, int m_up,
    int m_pad, int steps3, const float4* __restrict__ edec, float e1max, uint8_t* __restrict__ planes,
    float* __restrict__ sx, LinearSet zero) {
  constexpr int TQ = B / 4;
  __shared__ float xs[kMaxDecodeRows][B];
  __shared__ float red[4][kMaxDecodeRows][64];
  __shared__ int qv[kMaxDecodeRows][64];
  __shared__ float xmax[kMaxDecodeRows];
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int w = tid / 64;
  const int64_t b = blockIdx.y;
  const int64_t c_first = b * m_up / kBase3PerChunk;       // block b's first base-3 chunk
  const int64_t g0 = c_first * kBase3PerChunk + static_cast<int64_t>(blockIdx.x) * 64;
  const int o = static_cast<int>(g0 + lane - b * m_up);    // this lane's sample within block b
  const bool in_block = o >= 0 && o < m_up;
  constexpr int XPT = kMaxDecodeRows * B / kExpThreads;
  const int mb = m * B;
  uint32_t xr[XPT];
  const int k32 = static_cast<int>(k);
  if (xt == SDQ_F32) {
    const uint32_t* __restrict__ xp = static_cast<const uint32_t*>(x) + b * B;
#pragma unroll
    for (int r = 0; r < XPT; ++r) {
      if (kExpThreads * r >= mb) break;
      const int idx = tid + kExpThreads * r;
      xr[r] = idx < mb ? xp[(idx / B) * k32 + idx % B] : 0u;
    }
  } else {
    const uint16_t* __restrict__ xp = static_cast<const uint16_t*>(x) + b * B;
#pragma unroll
    for (int r = 0; r < XPT; ++r) {
      if (kExpThreads * r >= mb) break;
      const int idx = tid + kExpThreads * r;
      xr[r] = idx < mb ? xp[(idx / B) * k32 + idx % B] : 0u;
    }
  }
  float4 e[TQ / 4];
  const float4* ep = edec + static_cast<int64_t>(w * (TQ / 4)) * m_pad + (in_block ? o : 0);
#pragma unroll
  for (int q = 0; q < TQ / 4; ++q) e[q] = ep[static_cast<int64_t>(q) * m_pad];
#pragma unroll
  for (int r = 0; r < XPT; ++r) {
    if (kExpThreads * r >= mb) break;
    const int idx = tid + kExpThreads * r;
    if (idx < mb) {
      const float v = xt == SDQ_F32    ? __uint_as_float(xr[r])
                      : xt == SDQ_BF16 ? __uint_as_float(xr[r] << 16)
                                       : __half2float(__ushort_as_half(static_cast<unsigned short>(xr[r])));
      xs[idx / B][idx % B] = v;
    }
  }
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t n_wg = static_cast<int64_t>(gridDim.x) * gridDim.y;
  zero_outputs(zero, m, wg, n_wg, tid);
  __syncthreads();
  for (int i = w; i < m; i += 4) {
    float mx = 0.0f;
    for (int t = lane; t < B; t += 64) mx = fmaxf(mx, fabsf(xs[i][t]));
    mx = wave_max_nonneg(mx);
    if (lane == 0) xmax[i] = mx;
  }
  for (int i = 0; i < m; ++i) {
    const float4* xrow = reinterpret_cast<const float4*>(&xs[i][w * TQ]);
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
    for (int q = 0; q < TQ / 4; ++q) {
      const float4 v = xrow[q];
      a0 += e[q].x * v.x;
      a1 += e[q].y * v.y;
      a2 += e[q].z * v.z;
      a3 += e[q].w * v.w;
    }
    red[w][i][lane] = (a0 + a1) + (a2 + a3);
  }
  __syncthreads();
  for (int idx = tid; idx < m * 64; idx += kExpThreads) {
    const int i = idx / 64, l = idx % 64;
    const float val = (red[0][i][l] + red[1][i][l]) + (red[2][i][l] + red[3][i][l]);
    const float bound = xmax[i] * e1max;
    const int ol = static_cast<int>(g0 + l - b * m_up);
    qv[i][l] = bound > 0.0f && ol >= 0 && ol < m_up ? __float2int_rn(val * (kQ / bound)) : 0;
    if (blockIdx.x == 0 && l == 0) sx[static_cast<int64_t>(i) * nb + b] = bound / kQ;
  }
  __syncthreads();
  store_planes_b3(qv, m, npg, b, g0, c_first, steps3, planes);
}

// The plane expansions for fp16 and bf16 activations (the same plane layouts
// and side duties as expand_planes_kernel / expand_planes_b3_kernel), with the
// dot products on the matrix cores (planes_qv_mfma).  Grid: (slots, blocks /
// NB); NB = 2 only when M is a multiple of the code chunk (the blocks of a
// workgroup then use the same columns of E).
template <int B, int LEVELS, bool BF16, int NB>
__global__ __launch_bounds__(kExpThreads) void expand_planes_mfma_kernel(
    const void* __restrict__ x, int m, int npg, int64_t k, int64_t nb, int m_up, int cpb,
    const uint16_t* __restrict__ et_hi, const uint16_t* __restrict__ et_lo, float e1max,
    uint32_t* __restrict__ planes, float* __restrict__ sx, LinearSet zero) {
  __shared__ int qv[NB][kMaxDecodeRows][64];
  constexpr int kCpc = LEVELS == 2 ? 128 : 64;
  const int64_t b0 = static_cast<int64_t>(blockIdx.y) * NB;
  const int nbl = static_cast<int>(min<int64_t>(NB, nb - b0));
  const int64_t g0 = b0 * m_up / kCpc * kCpc + static_cast<int64_t>(blockIdx.x) * 64;
  planes_qv_mfma<B, BF16, NB>(static_cast<const uint16_t*>(x), m, static_cast<int>(k), b0, nbl, g0, m_up, nb,
                              blockIdx.x == 0, et_hi, et_lo, e1max, sx, qv);
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  zero_outputs(zero, m, wg, static_cast<int64_t>(gridDim.x) * gridDim.y, threadIdx.x);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    if (j >= nbl) break;
    store_planes<LEVELS>(qv[j], m, npg, (b0 + j) * cpb + static_cast<int64_t>(blockIdx.x) / (kCpc / 64),
                         static_cast<int>(blockIdx.x % (kCpc / 64)), planes);
  }
}

template <int B, bool BF16>
__global__ __launch_bounds__(kExpThreads) void expand_planes_b3_mfma_kernel(
    const void* __restrict__ x, int m, int npg, int64_t k, int64_t nb, int m_up, int steps3,
    const uint16_t* __restrict__ et_hi, const uint16_t* __restrict__ et_lo, float e1max,
    uint8_t* __restrict__ planes, float* __restrict__ sx, LinearSet zero) {
  __shared__ int qv[1][kMaxDecodeRows][64];
  const int64_t b = blockIdx.y;
  const int64_t c_first = b * m_up / kBase3PerChunk;
  const int64_t g0 = c_first * kBase3PerChunk + static_cast<int64_t>(blockIdx.x) * 64;
  planes_qv_mfma<B, BF16, 1>(static_cast<const uint16_t*>(x), m, static_cast<int>(k), b, 1, g0, m_up, nb,
                             blockIdx.x == 0, et_hi, et_lo, e1max, sx, qv);
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  zero_outputs(zero, m, wg, static_cast<int64_t>(gridDim.x) * gridDim.y, threadIdx.x);
  __syncthreads();
  store_planes_b3(qv[0], m, npg, b, g0, c_first, steps3, planes);
}

// One workgroup: one 64-row panel and 4 * bpw consecutive blocks, wave w
// taking blocks w * bpw .. w * bpw + bpw - 1 of them (the workgroup reads one
// contiguous stretch of the panel's chunks; consecutive workgroups continue
// it).  Per block, CH chunks per load batch; each chunk is loaded lane = row
// (1 KB per load), then a 4 x 4 transpose of 16-lane groups (permlane swaps)
// leaves word kg of row 16 cg + c in register cg of lane 16 kg + c: the B
// operand of the MFMA on column group cg.  The four waves' partial sums meet
// in LDS and leave with one atomic add (or store) per output.
template <int LEVELS, int NPG, int CH, bool M1>
__global__ __launch_bounds__(256) void gemv_mfma_kernel(
    LinearSet S, const uint4* __restrict__ planes, const float* __restrict__ sx, int m,
    int64_t n_chunks, int64_t nb, int m_up, int cpb, int bpw, int n_split, int accumulate) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  constexpr int SPC = LEVELS == 2 ? 2 : 1;          // k-steps per chunk
  constexpr int kCpc = LEVELS == 2 ? 128 : 64;
  __shared__ float red[4][NPG * 4][64];
  const int lane = threadIdx.x % 64;
  const int wave = threadIdx.x / 64;
  const int lin = linear_of(S, blockIdx.y);            // units: panels
  const int64_t panel = blockIdx.y - S.first[lin];
  const int64_t n = S.n[lin];
  const float* __restrict__ scales = S.scales[lin];
  float* __restrict__ y = S.y[lin];
  const int kg = lane / 16;
  const uint4* cbase = static_cast<const uint4*>(S.codes[lin]) + panel * n_chunks * kPanel + lane;
  float accf[NPG][4];
#pragma unroll
  for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) accf[pg][cg] = 0.0f;
  const int64_t b_begin = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * bpw;
  const int64_t b_end = min<int64_t>(nb, b_begin + bpw);
  for (int64_t b = b_begin; b < b_end; ++b) {
    v4i acc[NPG][4];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
      for (int cg = 0; cg < 4; ++cg) acc[pg][cg] = v4i{0, 0, 0, 0};
    const int64_t c_first = b * m_up / kCpc;        // block b's first code chunk
    // The block's plane scale of this lane's activation row of each group,
    // loaded now (unconditionally, from a clamped row: a load under a branch
    // is waited for on the spot) and used when the block ends.
    float sxv[NPG];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
      const int a = pg * 4 + kg;
      const float v = sx[static_cast<int64_t>(min(a, m - 1)) * nb + b];
      sxv[pg] = a < m ? v * (1.0f / kCodeScale<LEVELS>) : 0.0f;
    }
    for (int c0 = 0; c0 < cpb; c0 += CH) {
      uint4 q[CH];
      uint4 av[CH][SPC][NPG];
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        // A slot past the block's last (CH not dividing cpb) gets zero planes:
        // no branch, the accumulators stay in place.  Slots the block does not
        // reach hold zero planes; their code loads stay inside the layer.
        const bool live = c0 + j < cpb;
        const int jj = min(c0 + j, cpb - 1);
        q[j] = load_code_chunk(&cbase[min<int64_t>(c_first + jj, n_chunks - 1) * kPanel]);
        const int64_t slot = b * cpb + jj;
#pragma unroll
        for (int s = 0; s < SPC; ++s)
#pragma unroll
          for (int pg = 0; pg < NPG; ++pg) {
            if constexpr (M1) {   // compact planes: rows 0-2 stored, the rest zero
              const int p = lane % 16;
              const uint4 v = planes[(slot * SPC + s) * 12 + kg * 3 + min(p, 2)];
              av[j][s][pg] = live && p < 3 ? v : make_uint4(0u, 0u, 0u, 0u);
            } else {
              const uint4 v = planes[((slot * SPC + s) * NPG + pg) * 64 + lane];
              av[j][s][pg] = live ? v : make_uint4(0u, 0u, 0u, 0u);
            }
          }
      }
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        uint32_t r0 = q[j].x, r1 = q[j].y, r2 = q[j].z, r3 = q[j].w;
        {
          const auto s02 = __builtin_amdgcn_permlane32_swap(r0, r2, false, false);
          const auto s13 = __builtin_amdgcn_permlane32_swap(r1, r3, false, false);
          r0 = s02[0]; r2 = s02[1]; r1 = s13[0]; r3 = s13[1];
          const auto s01 = __builtin_amdgcn_permlane16_swap(r0, r1, false, false);
          const auto s23 = __builtin_amdgcn_permlane16_swap(r2, r3, false, false);
          r0 = s01[0]; r1 = s01[1]; r2 = s23[0]; r3 = s23[1];
        }
        const uint32_t wcg[4] = {r0, r1, r2, r3};
#pragma unroll
        for (int s = 0; s < SPC; ++s)
#pragma unroll
          for (int cg = 0; cg < 4; ++cg) {
            const uint32_t wv = wcg[cg];
            v4i bop;
#pragma unroll
            for (int di = 0; di < 4; ++di) {
              const int d = LEVELS == 2 ? 4 * s + di : di;
              bop[di] = code_bytes<LEVELS>(wv, d);
            }
#pragma unroll
            for (int pg = 0; pg < NPG; ++pg) {
              const uint4 a4 = av[j][s][pg];
              const v4i aop = {static_cast<int>(a4.x), static_cast<int>(a4.y), static_cast<int>(a4.z),
                               static_cast<int>(a4.w)};
              acc[pg][cg] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop, bop, acc[pg][cg], 0, 0, 0);
            }
          }
      }
    }
    // Block done: dequantise with the block's scale of this lane's activation row.
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
#pragma unroll
      for (int cg = 0; cg < 4; ++cg) {
        const float v = (static_cast<float>(acc[pg][cg][0]) * 65536.0f +
                         static_cast<float>(acc[pg][cg][1]) * 256.0f) +
                        static_cast<float>(acc[pg][cg][2]);
        accf[pg][cg] += sxv[pg] * v;
      }
    }
  }
  // Combine the four waves; output (pg, cg, lane): activation row 4 pg + lane / 16,
  // weight row 16 cg + lane % 16 of the panel.
#pragma unroll
  for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) red[wave][pg * 4 + cg][lane] = accf[pg][cg];
  __syncthreads();
  for (int idx = threadIdx.x; idx < NPG * 4 * 64; idx += 256) {
    const int pc = idx / 64, l = idx % 64;
    const int a = (pc / 4) * 4 + l / 16;
    const int64_t r = panel * kPanel + 16 * (pc % 4) + l % 16;
    if (a >= m || r >= n) continue;
    const float val = ((red[0][pc][l] + red[1][pc][l]) + (red[2][pc][l] + red[3][pc][l])) * scales[r];
    float* yp = &y[static_cast<int64_t>(a) * n + r];
    if (n_split > 1) unsafeAtomicAdd(yp, val);
    else *yp = accumulate ? *yp + val : val;
  }
}

// The same contraction with the planes shared through LDS: one workgroup owns
// four consecutive 64-row panels of one linear (one per wave) and bpg
// consecutive blocks; per block it copies the block's planes (cpb * NPG KB)
// into LDS once (global_load_lds, together with the first batch of code
// chunks: one round trip), and every wave contracts its own panel's codes
// against them,
// so each plane byte crosses L2 once per four panels instead of once per
// panel.  A wave adds its outputs into y itself (one atomic per output and
// workgroup when K is split).
template <int LEVELS, int NPG, int CH>
__global__ __launch_bounds__(256) void gemv_mfma_lds_kernel(
    LinearSet S, const uint4* __restrict__ planes, const float* __restrict__ sx, int m,
    int64_t n_chunks, int64_t nb, int m_up, int cpb, int bpg, int n_split, int accumulate) {
  extern __shared__ uint4 pls[];
  typedef int v4i __attribute__((ext_vector_type(4)));
  constexpr int SPC = LEVELS == 2 ? 2 : 1;
  constexpr int kCpc = LEVELS == 2 ? 128 : 64;
  const int lane = threadIdx.x % 64;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int lin = linear_of(S, blockIdx.y);            // units: groups of four panels
  const int64_t n = S.n[lin];
  const int64_t n_panels = (n + kPanel - 1) / kPanel;
  const int64_t panel = (blockIdx.y - S.first[lin]) * 4 + wave;
  const bool live = panel < n_panels;
  const float* __restrict__ scales = S.scales[lin];
  float* __restrict__ y = S.y[lin];
  const int kg = lane / 16;
  // A wave past the linear's last panel reads panel 0 (in bounds) and writes nothing.
  const uint4* __restrict__ cpanel =
      static_cast<const uint4*>(S.codes[lin]) + (live ? panel : 0) * n_chunks * kPanel;
  const int per_block = cpb * SPC * NPG * 64;           // uint4 of one block's planes
  float accf[NPG][4];
#pragma unroll
  for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) accf[pg][cg] = 0.0f;
  const int64_t b_begin = static_cast<int64_t>(blockIdx.x) * bpg;
  const int64_t b_end = min<int64_t>(nb, b_begin + bpg);
  for (int64_t b = b_begin; b < b_end; ++b) {
    const int64_t c_first = b * m_up / kCpc;
    // The block's first batch of code chunks, then its planes copied straight
    // into LDS (global_load_lds, 1 KB per wave and copy, all in flight at
    // once), then one wait for both.
    uint4 q[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) q[j] = load_code_chunk(&cpanel[min<int64_t>(c_first + j, n_chunks - 1) * kPanel + lane]);
    const uint4* __restrict__ src = planes + b * per_block;
    for (int i0 = wave * 64; i0 < per_block; i0 += 256)
      __builtin_amdgcn_global_load_lds((dec_gbl_ptr)(src + i0 + lane), (dec_lds_ptr)(pls + i0), 16, 0, 0);
    float sxv[NPG];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
      const int a = pg * 4 + kg;
      const float v = sx[static_cast<int64_t>(min(a, m - 1)) * nb + b];
      sxv[pg] = a < m ? v * (1.0f / kCodeScale<LEVELS>) : 0.0f;
    }
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();
    v4i acc[NPG][4];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
      for (int cg = 0; cg < 4; ++cg) acc[pg][cg] = v4i{0, 0, 0, 0};
    for (int c0 = 0; c0 < cpb; c0 += CH) {
      if (c0 > 0) {
#pragma unroll
        for (int j = 0; j < CH; ++j)
          q[j] = load_code_chunk(&cpanel[min<int64_t>(c_first + c0 + j, n_chunks - 1) * kPanel + lane]);
      }
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        uint32_t r0 = q[j].x, r1 = q[j].y, r2 = q[j].z, r3 = q[j].w;
        {
          const auto s02 = __builtin_amdgcn_permlane32_swap(r0, r2, false, false);
          const auto s13 = __builtin_amdgcn_permlane32_swap(r1, r3, false, false);
          r0 = s02[0]; r2 = s02[1]; r1 = s13[0]; r3 = s13[1];
          const auto s01 = __builtin_amdgcn_permlane16_swap(r0, r1, false, false);
          const auto s23 = __builtin_amdgcn_permlane16_swap(r2, r3, false, false);
          r0 = s01[0]; r1 = s01[1]; r2 = s23[0]; r3 = s23[1];
        }
        const uint32_t wcg[4] = {r0, r1, r2, r3};
#pragma unroll
        for (int s = 0; s < SPC; ++s)
#pragma unroll
          for (int cg = 0; cg < 4; ++cg) {
            const uint32_t wv = wcg[cg];
            v4i bop;
#pragma unroll
            for (int di = 0; di < 4; ++di) {
              const int d = LEVELS == 2 ? 4 * s + di : di;
              bop[di] = code_bytes<LEVELS>(wv, d);
            }
#pragma unroll
            for (int pg = 0; pg < NPG; ++pg) {
              const uint4 a4 = pls[(((c0 + j) * SPC + s) * NPG + pg) * 64 + lane];
              const v4i aop = {static_cast<int>(a4.x), static_cast<int>(a4.y), static_cast<int>(a4.z),
                               static_cast<int>(a4.w)};
              acc[pg][cg] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop, bop, acc[pg][cg], 0, 0, 0);
            }
          }
      }
    }
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
#pragma unroll
      for (int cg = 0; cg < 4; ++cg) {
        const float v = (static_cast<float>(acc[pg][cg][0]) * 65536.0f +
                         static_cast<float>(acc[pg][cg][1]) * 256.0f) +
                        static_cast<float>(acc[pg][cg][2]);
        accf[pg][cg] += sxv[pg] * v;
      }
    }
    __syncthreads();   // before the next block's planes overwrite these
  }
  if (!live) return;
  // output (pg, cg, lane): activation row 4 pg + lane / 16, weight row 16 cg + lane % 16
#pragma unroll
  for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) {
      const int a = pg * 4 + kg;
      const int64_t r = panel * kPanel + 16 * cg + lane % 16;
      if (a >= m || r >= n) continue;
      const float val = accf[pg][cg] * scales[r];
      float* yp = &y[static_cast<int64_t>(a) * n + r];
      if (n_split > 1) unsafeAtomicAdd(yp, val);
      else *yp = accumulate ? *yp + val : val;
    }
}

// The five base-3 digits d = code + 1 of each byte of w, as five words of
// four bytes (word j: digit j of bytes 0..3).  A byte q stores
// ceil(256 v / 243) for its digits' value v (first code most significant), so
// digit j is the integer part of 3 r, r the fraction left by the digits
// before it (r = q / 256 to begin with).  Bytes 0, 2 and 1, 3 travel as two
// 16-bit fractions per word; 3 r < 768 keeps each product inside its half,
// with the digit in the half's high byte: one v_perm gathers the four.
__device__ inline void base3_digits(uint32_t w, uint32_t d[5]) {
  uint32_t P = w & 0x00FF00FFu;           // bytes 0, 2
  uint32_t Q = (w >> 8) & 0x00FF00FFu;    // bytes 1, 3
#pragma unroll
  for (int j = 0; j < 5; ++j) {
    // 3 P as (P << 1) + P in one full-rate instruction (left to itself the
    // compiler turns it into a 24-bit multiply)
    asm("v_lshl_add_u32 %0, %1, 1, %1" : "=v"(P) : "v"(P));
    asm("v_lshl_add_u32 %0, %1, 1, %1" : "=v"(Q) : "v"(Q));
    d[j] = __builtin_amdgcn_perm(Q, P, 0x07030501u);   // P.b1 Q.b1 P.b3 Q.b3
    if (j < 4) {
      P &= 0x00FF00FFu;
      Q &= 0x00FF00FFu;
    }
  }
}

// gemv_mfma_kernel for base-3 codes: per group of four chunk slots, each
// slot's chunk is loaded lane = row and transposed as for 2-bit codes, its
// four bytes per lane give the digit bytes d = code + 1 of the slot's k-step
// and one word of the group's digit-4 k-step; the sums of d x less the sums
// of x (one more product per k-step against a B operand of ones) are the
// sums of code x.
template <int NPG>
__global__ __launch_bounds__(256) void gemv_mfma_b3_kernel(
    LinearSet S, const uint4* __restrict__ planes, const float* __restrict__ sx, int m,
    int64_t n_chunks, int64_t nb, int m_up, int cpb3, int steps3, int bpw, int n_split, int accumulate) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  __shared__ float red[4][NPG * 4][64];
  const int lane = threadIdx.x % 64;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int lin = linear_of(S, blockIdx.y);            // units: panels
  const int64_t panel = blockIdx.y - S.first[lin];
  const int64_t n = S.n[lin];
  const float* __restrict__ scales = S.scales[lin];
  float* __restrict__ y = S.y[lin];
  const int kg = lane / 16;
  const uint4* __restrict__ cpanel = static_cast<const uint4*>(S.codes[lin]) + panel * n_chunks * kPanel;
  const v4i ones = {0x01010101, 0x01010101, 0x01010101, 0x01010101};
  float accf[NPG][4];
#pragma unroll
  for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) accf[pg][cg] = 0.0f;
  const int64_t b_begin = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * bpw;
  const int64_t b_end = min<int64_t>(nb, b_begin + bpw);
  const int groups = steps3 / kB3Steps;
  for (int64_t b = b_begin; b < b_end; ++b) {
    v4i acc[NPG][4], acc1[NPG];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
      acc1[pg] = v4i{0, 0, 0, 0};
#pragma unroll
      for (int cg = 0; cg < 4; ++cg) acc[pg][cg] = v4i{0, 0, 0, 0};
    }
    const int64_t c_first = b * m_up / kBase3PerChunk;
    float sxv[NPG];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
      const int a = pg * 4 + kg;
      const float v = sx[static_cast<int64_t>(min(a, m - 1)) * nb + b];
      sxv[pg] = a < m ? v : 0.0f;
    }
    for (int G = 0; G < groups; ++G) {
      uint4 q[kB3Group];
      uint4 av[kB3Steps][NPG];
#pragma unroll
      for (int jj = 0; jj < kB3Group; ++jj)
        q[jj] = load_code_chunk(&cpanel[min<int64_t>(c_first + G * kB3Group + jj, n_chunks - 1) * kPanel + lane]);
#pragma unroll
      for (int st = 0; st < kB3Steps; ++st)
#pragma unroll
        for (int pg = 0; pg < NPG; ++pg)
          av[st][pg] = planes[((((b * steps3) + G * kB3Steps + st) * NPG + pg) * 64) + lane];
      uint32_t d4[4][kB3Group];
#pragma unroll
      for (int jj = 0; jj < kB3Group; ++jj) {
        // A slot past the block's last holds zero planes: its products are skipped.
        const bool live = G * kB3Group + jj < cpb3;
        uint32_t r0 = q[jj].x, r1 = q[jj].y, r2 = q[jj].z, r3 = q[jj].w;
        {
          const auto s02 = __builtin_amdgcn_permlane32_swap(r0, r2, false, false);
          const auto s13 = __builtin_amdgcn_permlane32_swap(r1, r3, false, false);
          r0 = s02[0]; r2 = s02[1]; r1 = s13[0]; r3 = s13[1];
          const auto s01 = __builtin_amdgcn_permlane16_swap(r0, r1, false, false);
          const auto s23 = __builtin_amdgcn_permlane16_swap(r2, r3, false, false);
          r0 = s01[0]; r1 = s01[1]; r2 = s23[0]; r3 = s23[1];
        }
        const uint32_t wcg[4] = {r0, r1, r2, r3};
#pragma unroll
        for (int cg = 0; cg < 4; ++cg) {
          uint32_t d[5];
          base3_digits(wcg[cg], d);
          d4[cg][jj] = d[4];
          if (live) {
            const v4i bop = {static_cast<int>(d[0]), static_cast<int>(d[1]), static_cast<int>(d[2]),
                             static_cast<int>(d[3])};
#pragma unroll
            for (int pg = 0; pg < NPG; ++pg) {
              const uint4 a4 = av[jj][pg];
              const v4i aop = {static_cast<int>(a4.x), static_cast<int>(a4.y), static_cast<int>(a4.z),
                               static_cast<int>(a4.w)};
              acc[pg][cg] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop, bop, acc[pg][cg], 0, 0, 0);
            }
          }
        }
        if (live) {
#pragma unroll
          for (int pg = 0; pg < NPG; ++pg) {
            const uint4 a4 = av[jj][pg];
            const v4i aop = {static_cast<int>(a4.x), static_cast<int>(a4.y), static_cast<int>(a4.z),
                             static_cast<int>(a4.w)};
            acc1[pg] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop, ones, acc1[pg], 0, 0, 0);
          }
        }
      }
      // the group's digit-4 step (a dead slot's word meets zero planes)
#pragma unroll
      for (int pg = 0; pg < NPG; ++pg) {
        const uint4 a4 = av[kB3Group][pg];
        const v4i aop = {static_cast<int>(a4.x), static_cast<int>(a4.y), static_cast<int>(a4.z),
                         static_cast<int>(a4.w)};
#pragma unroll
        for (int cg = 0; cg < 4; ++cg) {
          const v4i bop = {static_cast<int>(d4[cg][0]), static_cast<int>(d4[cg][1]), static_cast<int>(d4[cg][2]),
                           static_cast<int>(d4[cg][3])};
          acc[pg][cg] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop, bop, acc[pg][cg], 0, 0, 0);
        }
        acc1[pg] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop, ones, acc1[pg], 0, 0, 0);
      }
    }
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
#pragma unroll
      for (int cg = 0; cg < 4; ++cg) {
        const v4i t = acc[pg][cg] - acc1[pg];
        const float v = (static_cast<float>(t[0]) * 65536.0f + static_cast<float>(t[1]) * 256.0f) +
                        static_cast<float>(t[2]);
        accf[pg][cg] += sxv[pg] * v;
      }
    }
  }
#pragma unroll
  for (int pg = 0; pg < NPG; ++pg)
#pragma unroll
    for (int cg = 0; cg < 4; ++cg) red[wave][pg * 4 + cg][lane] = accf[pg][cg];
  __syncthreads();
  for (int idx = threadIdx.x; idx < NPG * 4 * 64; idx += 256) {
    const int pc = idx / 64, l = idx % 64;
    const int a = (pc / 4) * 4 + l / 16;
    const int64_t r = panel * kPanel + 16 * (pc % 4) + l % 16;
    if (a >= m || r >= n) continue;
    const float val = ((red[0][pc][l] + red[1][pc][l]) + (red[2][pc][l] + red[3][pc][l])) * scales[r];
    float* yp = &y[static_cast<int64_t>(a) * n + r];
    if (n_split > 1) unsafeAtomicAdd(yp, val);
    else *yp = accumulate ? *yp + val : val;
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = 0.0f;
}

// Byte K of x, masked with 60, in one instruction (a byte select on the
// operand): with x = w << 2 it is 4 times nibble 2K of w, with x = w >> 2 four
// times nibble 2K + 1.
template <int K>
__device__ inline uint32_t byte_and60(uint32_t x) {
  uint32_t r;
  if constexpr (K == 0)
    asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0" : "=v"(r) : "v"(x));
  else if constexpr (K == 1)
    asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1" : "=v"(r) : "v"(x));
  else if constexpr (K == 2)
    asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2" : "=v"(r) : "v"(x));
  else
    asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3" : "=v"(r) : "v"(x));
  return r;
}

template <int NIB>
__device__ inline uint32_t nibble_offset(uint32_t w4, uint32_t w2) {
  return byte_and60<NIB / 2>(NIB % 2 ? w2 : w4);
}

// Entries 4h .. 4h+3 of a 4-bit group's table.  Binary: bits b0..b3 of the
// entry select +x or -x for four consecutive samples; ternary: fields
// f0 = e & 3, f1 = e >> 2 weight two samples by {00: 0, 01: +1, 11: -1, 10: 0}.
template <int LEVELS>
__device__ inline float4 build_quad(const float (&xs)[4], int h) {
  float lo[4], hi;
  if (LEVELS == 2) {
    const float a0 = xs[0] + xs[1], a1 = xs[0] - xs[1];
    lo[0] = -a0; lo[1] = a1; lo[2] = -a1; lo[3] = a0;          // bits 1..0
    hi = ((h & 1) ? xs[2] : -xs[2]) + ((h & 2) ? xs[3] : -xs[3]);   // bits 3..2
  } else {
    lo[0] = 0.0f; lo[1] = xs[0]; lo[2] = 0.0f; lo[3] = -xs[0];
    hi = h == 1 ? xs[1] : (h == 3 ? -xs[1] : 0.0f);
  }
  return make_float4(lo[0] + hi, lo[1] + hi, lo[2] + hi, lo[3] + hi);
}

// One workgroup: one K segment of SEG chunks and four 64-row panels, one per
// wave (lane = weight row).  The workgroup first issues its loads -- the
// activation samples the tables need, then every lane's SEG code chunks
// (1 KB per wave and chunk, coalesced) -- then builds the segment's tables,
// shared by all four panels, and each lane adds one table entry per 4 bits of
// code per activation row.  Table offsets are compile-time constants, so a
// lookup costs a shift, a mask, an LDS read and an add.
template <int MR, int LEVELS, int SEG>
__global__ __launch_bounds__(64 * kGemvWaves) void gemv_lut_kernel(
    LinearSet S, const float* __restrict__ xt, int m, int64_t n_chunks,
    int64_t k_up_pad, int n_segs, int segs_fast, int accumulate) {
  constexpr int CPG = LEVELS == 2 ? 4 : 2;            // codes per 4-bit group
  constexpr int kGroups = SEG * kGroupsPerChunk;       // groups per activation row
  constexpr int kRowFloats = kGroups * 16;             // table floats per activation row
  constexpr int kThreads = 64 * kGemvWaves;
  constexpr int kEnt = MR * kRowFloats / kThreads;     // table entries built per thread
  constexpr int kGroupsPerThread = kEnt >= 16 ? kEnt / 16 : 1;
  constexpr int kSpan = kEnt >= 16 ? 16 : kEnt;        // entries per group built by a thread
  static_assert(kEnt >= 4 && kEnt % 4 == 0, "at least one float4 of table per thread");
  static_assert(MR * kRowFloats * 4 <= 65536, "table offsets fit the LDS immediate");
  __shared__ __attribute__((aligned(16))) float lut[MR * kRowFloats];

  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  const int64_t pg = segs_fast ? blockIdx.y : blockIdx.x;   // panel group over the set
  const int lin = linear_of(S, pg);                          // units: panel groups
  const int64_t n = S.n[lin];
  const int64_t n_panels = (n + kPanel - 1) / kPanel;
  const uint4* __restrict__ codes = static_cast<const uint4*>(S.codes[lin]);
  const float* __restrict__ scales = S.scales[lin];
  float* __restrict__ y = S.y[lin];
  const int64_t panel = (pg - S.first[lin]) * kGemvWaves + wave;
  const bool panel_ok = panel < n_panels;
  const int seg = segs_fast ? blockIdx.x : blockIdx.y;
  const int64_t c0 = static_cast<int64_t>(seg) * SEG;
  const int nch = static_cast<int>(min<int64_t>(SEG, n_chunks - c0));
  const int64_t code0 = c0 * kGroupsPerChunk * CPG;   // first code of the segment

  // 1. Loads: the samples of this thread's table groups first, then the code
  //    chunks (vector memory returns in order: the build waits only for the
  //    samples while the code stream is in flight).
  float4 xv[kGroupsPerThread];
  int grow[kGroupsPerThread], ggrp[kGroupsPerThread];
  bool gok[kGroupsPerThread];
  const int e0 = (tid * kEnt) % 16;
#pragma unroll
  for (int gi = 0; gi < kGroupsPerThread; ++gi) {
    const int f = tid * kEnt + gi * 16;                // first table float of the group
    grow[gi] = f / kRowFloats;
    ggrp[gi] = (f % kRowFloats) / 16;
    gok[gi] = grow[gi] < m && ggrp[gi] < nch * kGroupsPerChunk;
    const float* xp = xt + (gok[gi] ? static_cast<int64_t>(grow[gi]) * k_up_pad + code0 + ggrp[gi] * CPG : 0);
    if (CPG == 4) {
      xv[gi] = *reinterpret_cast<const float4*>(xp);
    } else {
      const float2 v = *reinterpret_cast<const float2*>(xp);
      xv[gi] = make_float4(v.x, v.y, 0.f, 0.f);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  uint4 q[SEG];
  {
    const uint4* src = codes + ((panel_ok ? panel : n_panels - 1) * n_chunks + c0) * kPanel + lane;
#pragma unroll
    for (int j = 0; j < SEG; ++j) q[j] = load_code_chunk(&src[static_cast<int64_t>(min(j, nch - 1)) * kPanel]);
  }
  __builtin_amdgcn_sched_barrier(0);

  // 2. Tables: 16 entries per (activation row, group); groups past the
  //    segment end and rows >= m are all zero.
#pragma unroll
  for (int gi = 0; gi < kGroupsPerThread; ++gi) {
    const float4 v = xv[gi];
    const bool ok = gok[gi];
    const float xs[4] = {ok ? v.x : 0.f, ok ? v.y : 0.f, ok ? v.z : 0.f, ok ? v.w : 0.f};
    float* dst = lut + grow[gi] * kRowFloats + ggrp[gi] * 16 + e0;
#pragma unroll
    for (int e = 0; e < kSpan; e += 4)
      *reinterpret_cast<float4*>(dst + e) = build_quad<LEVELS>(xs, (e0 + e) / 4);
  }
  __builtin_amdgcn_sched_barrier(0);     // the table is written before any code word is waited for
  __syncthreads();

  // 3. Lookups.
  float acc[MR];
#pragma unroll
  for (int i = 0; i < MR; ++i) acc[i] = 0.0f;
  const char* lbytes = reinterpret_cast<const char*>(lut);
#pragma unroll
  for (int c = 0; c < SEG; ++c) {
    const uint32_t words[4] = {q[c].x, q[c].y, q[c].z, q[c].w};
#pragma unroll
    for (int wi = 0; wi < 4; ++wi) {
      // byte offset of entry e = nibble value: 4 * e
      const uint32_t w4 = words[wi] << 2, w2 = words[wi] >> 2;
      const uint32_t offs[8] = {nibble_offset<0>(w4, w2), nibble_offset<1>(w4, w2), nibble_offset<2>(w4, w2),
                                nibble_offset<3>(w4, w2), nibble_offset<4>(w4, w2), nibble_offset<5>(w4, w2),
                                nibble_offset<6>(w4, w2), nibble_offset<7>(w4, w2)};
#pragma unroll
      for (int nib = 0; nib < 8; ++nib) {
#pragma unroll
        for (int i = 0; i < MR; ++i)
          acc[i] += *reinterpret_cast<const float*>(lbytes + (i * kRowFloats + (c * kGroupsPerChunk + wi * 8 + nib) * 16) * 4 + offs[nib]);
      }
      // Make each word's sums complete before the next word's table reads
      // (otherwise the compiler sinks the adds and keeps every read live:
      // register pressure).
#pragma unroll
      for (int i = 0; i < MR; ++i) asm volatile("" : "+v"(acc[i]));
    }
  }

  // 4. Scale and write: a plain store (or add) when the segment is the whole
  //    row, otherwise an atomic add into y (zeroed beforehand, or holding the
  //    values to accumulate onto).
  const int64_t r = panel * kPanel + lane;
  // A use of the code registers on every lane: otherwise the compiler sinks
  // the code loads into the live-lane branch below, past the table build and
  // its barrier, and the code stream starts only after the tables are built.
#pragma unroll
  for (int c = 0; c < SEG; ++c) asm volatile("" ::"v"(q[c].x));
  if (!panel_ok || r >= n) return;
  const float s = scales[r];
#pragma unroll
  for (int i = 0; i < MR; ++i) {
    if (i >= m) break;
    float* yp = &y[static_cast<int64_t>(i) * n + r];
    if (n_segs > 1) unsafeAtomicAdd(yp, acc[i] * s);
    else *yp = accumulate ? *yp + acc[i] * s : acc[i] * s;
  }
}

// 4 * ((x >> 8) & 255) in one instruction (a byte select on the shifted operand).
__device__ inline uint32_t byte1_times4(uint32_t x) {
  uint32_t r;
  asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
      : "=v"(r) : "v"(x));
  return r;
}

// Base-3 codes (one activation row): byte p of a chunk holds codes 5p .. 5p+4
// as q = ceil(256 v / 243), v = 81 d0 + 27 d1 + 9 d2 + 3 d3 + d4 (d = code + 1).
// Per byte two tables: 27 entries for its first three codes, indexed by
// 9 d0 + 3 d1 + d2 = (27 q) >> 8, and 9 for its last two, indexed by
// 3 d3 + d4 = (9 ((27 q) & 255)) >> 8 (both exact for every stored byte):
// a multiply and a byte select each.  Each table spans at most 27
// consecutive words, so a wave's reads of one table hit distinct banks or
// the same word.  Otherwise as the 2-bit table GEMV: loads first, tables of
// the segment shared by four panels, one wave per panel.
template <int SEG>
__global__ __launch_bounds__(64 * kGemvWaves) void gemv_lut_base3_kernel(
    LinearSet S, const float* __restrict__ xt, int64_t n_chunks, int n_segs, int segs_fast,
    int accumulate) {
  constexpr int kBytes = 16;                   // groups of five codes per chunk
  constexpr int kGF = 36;                      // table floats per group: 27 + 9
  constexpr int kGroups = SEG * kBytes;
  constexpr int kThreads = 64 * kGemvWaves;
  static_assert(2 * kGroups <= kThreads, "one table per thread at most");
  static_assert(kGroups * kGF * 4 <= 65536, "table offsets fit the LDS immediate");
  __shared__ __attribute__((aligned(16))) float lut[kGroups * kGF];

  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  const int64_t pg = segs_fast ? blockIdx.y : blockIdx.x;   // panel group over the set
  const int lin = linear_of(S, pg);
  const int64_t n = S.n[lin];
  const int64_t n_panels = (n + kPanel - 1) / kPanel;
  const uint4* __restrict__ codes = static_cast<const uint4*>(S.codes[lin]);
  const float* __restrict__ scales = S.scales[lin];
  float* __restrict__ y = S.y[lin];
  const int64_t panel = (pg - S.first[lin]) * kGemvWaves + wave;
  const bool panel_ok = panel < n_panels;
  const int seg = segs_fast ? blockIdx.x : blockIdx.y;
  const int64_t c0 = static_cast<int64_t>(seg) * SEG;
  const int nch = static_cast<int>(min<int64_t>(SEG, n_chunks - c0));
  const int64_t code0 = c0 * kBase3PerChunk;

  // 1. Loads.  Threads [0, kGroups) build the 27-entry tables (samples
  //    5g .. 5g+2), threads [kGroups, 2 kGroups) the 9-entry ones (5g+3, 5g+4);
  //    xs = {the two low-order samples, the leading one}.
  const bool is_lo = tid < kGroups;
  const int g = is_lo ? tid : tid - kGroups;
  const bool gok = tid < 2 * kGroups && g < nch * kBytes;
  float xs[3] = {0.f, 0.f, 0.f};
  if (gok) {
    const float* xp = xt + code0 + 5 * g + (is_lo ? 1 : 3);
    xs[0] = xp[0];
    xs[1] = xp[1];
    if (is_lo) xs[2] = xp[-1];
  }
  __builtin_amdgcn_sched_barrier(0);
  uint4 q[SEG];
  {
    const uint4* src = codes + ((panel_ok ? panel : n_panels - 1) * n_chunks + c0) * kPanel + lane;
#pragma unroll
    for (int j = 0; j < SEG; ++j) q[j] = load_code_chunk(&src[static_cast<int64_t>(min(j, nch - 1)) * kPanel]);
  }
  __builtin_amdgcn_sched_barrier(0);

  // 2. Tables: entry (9 c +) 3 a + b = ((c - 1) xs[2] +) (a - 1) xs[0] + (b - 1) xs[1].
  if (tid < 2 * kGroups) {
    float* dst = lut + g * kGF + (is_lo ? 0 : 27);
    float t9[9];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 3; ++b) t9[3 * a + b] = static_cast<float>(a - 1) * xs[0] + static_cast<float>(b - 1) * xs[1];
    if (is_lo) {
#pragma unroll
      for (int c = 0; c < 3; ++c)
#pragma unroll
        for (int e = 0; e < 9; ++e) dst[9 * c + e] = t9[e] + static_cast<float>(c - 1) * xs[2];
    } else {
#pragma unroll
      for (int e = 0; e < 9; ++e) dst[e] = t9[e];
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();

  // 3. Lookups: two per byte.
  float acc = 0.0f;
#pragma unroll
  for (int c = 0; c < SEG; ++c) {
    const uint32_t words[4] = {q[c].x, q[c].y, q[c].z, q[c].w};
#pragma unroll
    for (int wi = 0; wi < 4; ++wi) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t t = ((words[wi] >> (8 * k)) & 255u) * 27u;
        const uint32_t lead4 = byte1_times4(t);                   // 4 ((27 q) >> 8)
        const uint32_t tail4 = byte1_times4((t & 255u) * 9u);     // 4 ((9 ((27 q) & 255)) >> 8)
        const char* tg = reinterpret_cast<const char*>(lut + (c * kBytes + wi * 4 + k) * kGF);
        acc += *reinterpret_cast<const float*>(tg + lead4);
        acc += *reinterpret_cast<const float*>(tg + 27 * 4 + tail4);
      }
      asm volatile("" : "+v"(acc));
    }
  }

  // 4. Scale and write (as the 2-bit table GEMV).
  const int64_t r = panel * kPanel + lane;
#pragma unroll
  for (int c = 0; c < SEG; ++c) asm volatile("" ::"v"(q[c].x));
  if (!panel_ok || r >= n) return;
  const float s = scales[r];
  if (n_segs > 1) unsafeAtomicAdd(&y[r], acc * s);
  else y[r] = accumulate ? y[r] + acc * s : acc * s;
}

int round_mr(int64_t m) {
  if (m <= 1) return 1;
  if (m <= 2) return 2;
  if (m <= 4) return 4;
  if (m <= 8) return 8;
  return 16;
}

// Chunks per K segment of the table GEMV.  Each segment adds one atomic per
// output into y, and the atomics on one address serialise, so the segments
// per output (n_chunks / SEG) set a floor; smaller segments give more
// workgroups to stream the codes.  Measured on MI355X at m = 1 over nine layer
// shapes (768 x 768 to 28672 x 8192 and 8192 x 28672): SEG = 4 is best unless
// it leaves fewer than 800 workgroups and SEG = 2 keeps the segments per
// output at 80 or below (small layers: 2), or it needs more than 128 segments
// per output (long rows: 8).  Tables of MR rows x SEG chunks must fit 64 KB.
// `panels`: the 64-row panels of all linears the launch covers.
int pick_seg(const sdq_layout* L, int mr, int64_t panels) {
  static const char* env = std::getenv("SDQ_GEMV_SEG");   // tuning aid: 2, 4 or 8
  const int max_seg = mr >= 16 ? 2 : (mr >= 8 ? 4 : 8);
  if (env) {
    const int v = std::atoi(env);
    if ((v == 2 || v == 4 || v == 8) && v <= max_seg) return v;
  }
  const int64_t panel_groups = (panels + kGemvWaves - 1) / kGemvWaves;
  const int64_t segs2 = (L->n_chunks + 1) / 2, segs4 = (L->n_chunks + 3) / 4;
  int seg;
  if (segs2 <= 80 && panel_groups * segs4 < 800) seg = 2;
  else if (segs4 > 128) seg = 8;
  else seg = 4;
  return std::min(seg, max_seg);
}

int segs_for(const sdq_layout* L, int seg) {
  return static_cast<int>((L->n_chunks + seg - 1) / seg);
}

// Decode variants: 2..16 rows run the integer-MFMA contraction, whose cost
// hardly grows with the row count; one row of ternary 2-bit fields runs it
// too on long upsampled rows (compact planes, three operand rows of
// sixteen), short rows and binary and base-3 codes the addition-only table
// GEMV (the plane expansion costs ~0.5 us more than the table path's, which
// the faster contraction repays from ~40 MB of codes per call).  Measured on
// MI355X at m = 1 (70B shapes, expansion + contraction in graph replay):
// gate/up OSR 3 69.3 -> 66.2 us, OSR 2 49.4 -> 47.7, down OSR 3 41.3 -> 40.4,
// q/k/v OSR 3 19.8 -> 19.6 but OSR 1.5 12.1 -> 13.3; the LLaMA-7B binary
// down_proj 8.2 -> 10.3 and base-3 gate/up 62.6 -> 140 us.  The rule depends
// on the layout's k, M, levels and packing only, which the linears of one
// group share.  SDQ_DECODE_PATH=lut or =mfma forces one (a tuning and
// cross-check aid, read on every call).
constexpr int64_t kMfmaRowKup = 16384;   // one row: the MFMA path from k * M / B samples
bool use_mfma(const sdq_layout* L, int64_t m) {
  const char* env = std::getenv("SDQ_DECODE_PATH");
  if (env && std::string(env) == "lut") return false;
  if (env && std::string(env) == "mfma") return true;
  return m >= 2 || (L->levels == 3 && L->packing == SDQ_PACK_FIELDS && L->k_up >= kMfmaRowKup);
}

int npg_for(int64_t m) { return static_cast<int>((m + 3) / 4); }

// Chunk slots per block in the plane layout: the most code chunks any block
// touches (M / chunk when blocks start on chunks).
int mfma_cpb(const sdq_layout* L) {
  const int64_t cpc = L->levels == 2 ? 128 : 64;
  int64_t most = 0;
  for (int64_t b = 0; b < L->nb; ++b) {
    const int64_t first = b * L->m_up / cpc;
    const int64_t end = ((b + 1) * L->m_up + cpc - 1) / cpc;
    most = std::max(most, end - first);
    if (L->m_up % cpc == 0) break;                 // every block alike
  }
  return static_cast<int>(most);
}

// Base-3 chunk slots per block on the MFMA path (the most 80-code chunks any
// block touches, rounded up to whole groups of four) and k-steps per block.
int mfma_cpb3(const sdq_layout* L) {
  int64_t most = 0;
  for (int64_t b = 0; b < L->nb; ++b) {
    const int64_t first = b * L->m_up / kBase3PerChunk;
    const int64_t end = ((b + 1) * L->m_up + kBase3PerChunk - 1) / kBase3PerChunk;
    most = std::max(most, end - first);
    if (L->m_up % kBase3PerChunk == 0) break;
  }
  return static_cast<int>(most);
}
int mfma_steps3(const sdq_layout* L) { return (mfma_cpb3(L) + kB3Group - 1) / kB3Group * kB3Steps; }
bool mfma_base3(const sdq_layout* L, int64_t m) { return L->packing == SDQ_PACK_BASE3 && use_mfma(L, m); }

int pick_ch(int cpb, int npg, int levels);
constexpr int64_t kLdsPlanesWgs = 768;

// Whether a 2-16-row contraction over `panels` panels shares its planes
// through LDS (gemv_mfma_lds_kernel): for two or three plane groups (5-12
// rows) on launches of at least kLdsPlanesWgs workgroups of four panels
// (at one block per wave), when the chunks go in batches of four or the rows
// are long (64 blocks or more).  Measured on MI355X at m = 8 (70B shapes):
// gate/up 93 -> 87 us at OSR 3 and 65 -> 62 us at OSR 2 (batches of four),
// but 78 -> 80 at OSR 2.5 and 51 -> 53 at 1.5 (batches of two); down 2-6 %
// faster at OSR 1.5-3; the smaller q/k/v and o launches (256-320 workgroups
// of four panels) ran 21 -> 31 and 17 -> 27 us.  At m = 12 (planes copied
// with global_load_lds): gate/up 108 -> 89 us at OSR 3, down 59 -> 50.  Four
// plane groups were slower at every size (m = 16 gate/up 136 -> 144 us).
// SDQ_MFMA_LDS=0 or 1 forces the choice (a tuning and test aid, read on every
// call so that a test can take both paths in one process).
bool mfma_lds(const sdq_layout* L, int64_t m, int64_t panels) {
  const int npg = npg_for(m);
  if (mfma_base3(L, m) || (npg != 2 && npg != 3)) return false;
  const size_t lds_bytes = static_cast<size_t>(mfma_cpb(L)) * (L->levels == 2 ? 2 : 1) * npg * 1024;
  if (lds_bytes > 65536) return false;
  const char* env = std::getenv("SDQ_MFMA_LDS");
  if (env && (std::atoi(env) == 0 || std::atoi(env) == 1)) return std::atoi(env) == 1;
  const int64_t splits1 = (L->nb + 3) / 4;
  const int ch = pick_ch(mfma_cpb(L), npg, L->levels);
  return splits1 * ((panels + kGemvWaves - 1) / kGemvWaves) >= kLdsPlanesWgs && (ch >= 4 || L->nb >= 64);
}

// Blocks per wave of the MFMA GEMV (each split over K costs one atomic add per
// output); SDQ_MFMA_BPW overrides.  Measured on MI355X (70B shapes and
// 8192 x 8192, OSR 2): one block per wave is best up to two plane groups
// (m <= 8) and on the LDS-shared launches; otherwise, from three plane groups
// on, the longer-lived waves of two blocks each win (m = 16: 64 -> 56 us on
// 28672 x 8192, 72 -> 59 us on 8192 x 28672; m = 12 o_proj 21.7 -> 19.5 us).
int mfma_bpw(const sdq_layout* L, int64_t m, int64_t panels) {
  static const char* env = std::getenv("SDQ_MFMA_BPW");
  if (env) {
    const int v = std::atoi(env);
    if (v >= 1) return v;
  }
  const int npg = npg_for(m);
  if (npg <= 2) return 1;
  return npg == 3 && mfma_lds(L, m, panels) ? 1 : 2;
}

// Workgroups along K per panel (each covers 4 * bpw blocks).
int mfma_splits(const sdq_layout* L, int64_t m, int64_t panels) {
  const int bpw = mfma_bpw(L, m, panels);
  return static_cast<int>((L->nb + 4 * bpw - 1) / (4 * bpw));
}

struct DecodeWs {
  float* xt;          // table path: x_tilde, m x k_up_pad fp32
  uint32_t* planes;   // MFMA path: fixed-point planes, nb x cpb x (chunk / 64) k-steps x npg x 1 KB
                      // (one row: 192 bytes per k-step)
  float* sx;          // MFMA path: per (row, block) plane scale, m x nb fp32
  size_t bytes;
};

// Workspace: the expansion output at offset 0, so one expansion can serve
// several linears that share its (k, block, M, levels).
DecodeWs carve(const sdq_layout* L, int64_t m, void* base) {
  DecodeWs w{};
  char* p = static_cast<char*>(base);
  if (use_mfma(L, m)) {
    const size_t steps = mfma_base3(L, m) ? static_cast<size_t>(L->nb) * mfma_steps3(L)
                                          : static_cast<size_t>(L->nb) * mfma_cpb(L) * (L->levels == 2 ? 2 : 1);
    // (one activation row of 2-bit fields: compact planes, 192 bytes per k-step)
    const size_t per_step = m == 1 && !mfma_base3(L, m) ? 192 : static_cast<size_t>(npg_for(m)) * 1024;
    const size_t pl = align_up(steps * per_step, 256);
    w.planes = reinterpret_cast<uint32_t*>(p);
    w.sx = reinterpret_cast<float*>(p + pl);
    w.bytes = pl + align_up(static_cast<size_t>(m) * L->nb * 4, 256);
  } else {
    const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
    w.xt = reinterpret_cast<float*>(p);
    w.bytes = align_up(static_cast<size_t>(m) * k_up_pad * 4, 256);
  }
  return w;
}

// Chunks loaded per batch: the largest allowed size that divides the block's
// chunks (all of them at once when they fit), within a register budget that
// shrinks with the number of plane groups.  For one plane group (1-4 rows),
// when that takes more than twice the fewest batches the budget allows (a
// prime chunk count, say), the batches are balanced instead and the last one
// carries a few dead slots (zero planes): measured on MI355X at m = 1, 11
// chunks per block (OSR 2.75) had gone in 11 batches of one, the waves
// waiting for memory 74 % of the time; 70B gate/up 54.9 -> 53.3 us, down
// 29.6 -> 28.8, q/k/v 13.1 -> 12.8.  With two plane groups the same rule
// measured slower (m = 8 q/k/v 16.9 -> 19.1 us), and the LDS kernel takes
// divisors only.
int pick_ch(int cpb, int npg, int levels) {
  const int cap_steps = npg == 1 ? 16 : (npg == 2 ? 8 : 4);
  const int cap = std::max(1, cap_steps / (levels == 2 ? 2 : 1));
  static const int allowed1[] = {8, 6, 4, 3, 2, 1};
  static const int allowed2[] = {4, 2, 1};
  const int* al = npg == 1 ? allowed1 : allowed2;
  const int na = npg == 1 ? 6 : 3;
  int div = 1, maxch = 1;
  for (int i = na - 1; i >= 0; --i) {
    if (al[i] > cap) continue;
    maxch = al[i];
    if (cpb % al[i] == 0) div = al[i];
  }
  const int fewest = (cpb + maxch - 1) / maxch;
  if (npg > 1 || (cpb + div - 1) / div <= 2 * fewest) return div;
  const int need = (cpb + fewest - 1) / fewest;
  for (int i = na - 1; i >= 0; --i)
    if (al[i] <= cap && al[i] >= need) return al[i];
  return maxch;
}

// Prefix sums of a set's units: `per(n)` units for a linear of n rows.
template <typename F>
int64_t fill_first(LinearSet& S, F per) {
  S.first[0] = 0;
  for (int j = 0; j < S.count; ++j) S.first[j + 1] = S.first[j] + per(S.n[j]);
  for (int j = S.count + 1; j <= kMaxGroup; ++j) S.first[j] = S.first[S.count];
  return S.first[S.count];
}

int64_t panels_of(int64_t n) { return (n + kPanel - 1) / kPanel; }
int64_t pgroups_of(int64_t n) { return (panels_of(n) + kGemvWaves - 1) / kGemvWaves; }

template <int LEVELS, int NPG, int CH, bool M1 = false>
void launch_mfma_ch(const DecodeWs& w, LinearSet S, const sdq_layout* L, int64_t m, bool accumulate,
                    hipStream_t stream) {
  const int64_t panels = fill_first(S, panels_of);
  const int bpw = mfma_bpw(L, m, panels);
  const int splits = mfma_splits(L, m, panels);
  if constexpr (!M1 && (NPG == 2 || NPG == 3)) {
    if (mfma_lds(L, m, panels)) {
      LinearSet S4 = S;
      const int64_t pgroups = fill_first(S4, pgroups_of);
      const size_t lds_bytes = static_cast<size_t>(mfma_cpb(L)) * (LEVELS == 2 ? 2 : 1) * NPG * 1024;
      const dim3 grid4(static_cast<unsigned>(splits), static_cast<unsigned>(pgroups));
      gemv_mfma_lds_kernel<LEVELS, NPG, CH><<<grid4, dim3(256), lds_bytes, stream>>>(
          S4, reinterpret_cast<const uint4*>(w.planes), w.sx, static_cast<int>(m), L->n_chunks, L->nb,
          L->m_up, mfma_cpb(L), 4 * bpw, splits, accumulate ? 1 : 0);
      return;
    }
  }
  // K groups fastest: consecutive workgroups sweep one panel's chunks.
  const dim3 grid(static_cast<unsigned>(splits), static_cast<unsigned>(panels));
  gemv_mfma_kernel<LEVELS, NPG, CH, M1><<<grid, dim3(256), 0, stream>>>(
      S, reinterpret_cast<const uint4*>(w.planes), w.sx, static_cast<int>(m), L->n_chunks, L->nb, L->m_up,
      mfma_cpb(L), bpw, splits, accumulate ? 1 : 0);
}

template <int LEVELS>
void launch_mfma_levels(const DecodeWs& w, const LinearSet& S, const sdq_layout* L, int64_t m, bool acc,
                        hipStream_t stream) {
  const int npg = npg_for(m);
  const int ch = pick_ch(mfma_cpb(L), npg, LEVELS);
#define SDQ_CH(NPG_, CH_)                                                         \
  if (ch == CH_) return launch_mfma_ch<LEVELS, NPG_, CH_>(w, S, L, m, acc, stream)
#define SDQ_CH1(CH_)                                                              \
  if (ch == CH_) return launch_mfma_ch<LEVELS, 1, CH_, true>(w, S, L, m, acc, stream)
  if (m == 1) {   // compact planes
    SDQ_CH1(8); SDQ_CH1(6); SDQ_CH1(4); SDQ_CH1(3); SDQ_CH1(2);
    return launch_mfma_ch<LEVELS, 1, 1, true>(w, S, L, m, acc, stream);
  }
#undef SDQ_CH1
  switch (npg) {
    case 1:
      SDQ_CH(1, 8); SDQ_CH(1, 6); SDQ_CH(1, 4); SDQ_CH(1, 3); SDQ_CH(1, 2);
      return launch_mfma_ch<LEVELS, 1, 1>(w, S, L, m, acc, stream);
    case 2:
      SDQ_CH(2, 4); SDQ_CH(2, 2);
      return launch_mfma_ch<LEVELS, 2, 1>(w, S, L, m, acc, stream);
    case 3:
      SDQ_CH(3, 4); SDQ_CH(3, 2);
      return launch_mfma_ch<LEVELS, 3, 1>(w, S, L, m, acc, stream);
    default:
      SDQ_CH(4, 4); SDQ_CH(4, 2);
      return launch_mfma_ch<LEVELS, 4, 1>(w, S, L, m, acc, stream);
  }
#undef SDQ_CH
}

// Large launches: segments fastest, so consecutive workgroups sweep the same
// panels' chunks.  Small ones (the whole grid resident at once): panel groups
// fastest, so neighbours share a segment's samples.  (Measured.)
dim3 lut_grid(int64_t pgroups, int n_segs, bool* segs_fast) {
  *segs_fast = pgroups * n_segs > 2048;
  return *segs_fast ? dim3(static_cast<unsigned>(n_segs), static_cast<unsigned>(pgroups))
                    : dim3(static_cast<unsigned>(pgroups), static_cast<unsigned>(n_segs));
}

template <int MR, int LEVELS, int SEG>
void launch_gemv_seg(const DecodeWs& w, LinearSet S, const sdq_layout* L, int64_t m, bool accumulate,
                     hipStream_t stream) {
  const int64_t pgroups = fill_first(S, pgroups_of);
  const int n_segs = segs_for(L, SEG);
  bool segs_fast = false;
  const dim3 grid = lut_grid(pgroups, n_segs, &segs_fast);
  gemv_lut_kernel<MR, LEVELS, SEG><<<grid, dim3(64 * kGemvWaves), 0, stream>>>(
      S, w.xt, static_cast<int>(m), L->n_chunks, L->n_chunks * L->codes_per_chunk, n_segs, segs_fast ? 1 : 0,
      accumulate ? 1 : 0);
}

template <int SEG>
void launch_gemv_base3_seg(const DecodeWs& w, LinearSet S, const sdq_layout* L, bool accumulate,
                           hipStream_t stream) {
  const int64_t pgroups = fill_first(S, pgroups_of);
  const int n_segs = segs_for(L, SEG);
  bool segs_fast = false;
  const dim3 grid = lut_grid(pgroups, n_segs, &segs_fast);
  gemv_lut_base3_kernel<SEG><<<grid, dim3(64 * kGemvWaves), 0, stream>>>(
      S, w.xt, L->n_chunks, n_segs, segs_fast ? 1 : 0, accumulate ? 1 : 0);
}

template <int MR, int LEVELS>
void launch_gemv_mr(const DecodeWs& w, const LinearSet& S, const sdq_layout* L, int64_t m, bool acc,
                    hipStream_t stream) {
  const int seg = pick_seg(L, MR, set_panels(S));
  if constexpr (MR <= 4) {
    if (seg == 8) return launch_gemv_seg<MR, LEVELS, 8>(w, S, L, m, acc, stream);
  }
  if constexpr (MR <= 8) {
    if (seg == 4) return launch_gemv_seg<MR, LEVELS, 4>(w, S, L, m, acc, stream);
  }
  launch_gemv_seg<MR, LEVELS, 2>(w, S, L, m, acc, stream);
}

template <int LEVELS>
void launch_gemv(const DecodeWs& w, const LinearSet& S, const sdq_layout* L, int64_t m, bool acc,
                 hipStream_t stream) {
  switch (round_mr(m)) {
    case 1: launch_gemv_mr<1, LEVELS>(w, S, L, m, acc, stream); break;
    case 2: launch_gemv_mr<2, LEVELS>(w, S, L, m, acc, stream); break;
    case 4: launch_gemv_mr<4, LEVELS>(w, S, L, m, acc, stream); break;
    case 8: launch_gemv_mr<8, LEVELS>(w, S, L, m, acc, stream); break;
    default: launch_gemv_mr<16, LEVELS>(w, S, L, m, acc, stream); break;
  }
}

}  // namespace

size_t decode_ws_bytes(const sdq_layout* L, int64_t m) { return carve(L, m, nullptr).bytes; }

sdq_status decode_supported(const sdq_layout* L) {
  (void)L;
  return SDQ_OK;
}

bool decode_reads_base3(const sdq_layout* L, int64_t m) {
  return L->packing == SDQ_PACK_BASE3 && (m == 1 || use_mfma(L, m));
}

bool decode_needs_zero_y(const sdq_layout* L, int64_t m, int64_t panels) {
  if (use_mfma(L, m)) return mfma_splits(L, m, panels) > 1;
  return segs_for(L, pick_seg(L, round_mr(m), panels)) > 1;
}

sdq_status launch_decode_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                const Tables* T, void* ws, const LinearSet* zero, hipStream_t stream) {
  const DecodeWs w = carve(L, m, ws);
  const int B = L->block;
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const LinearSet z = zero ? *zero : LinearSet{};
  const dim3 egrid(static_cast<unsigned>(T->m_pad / 64), static_cast<unsigned>(L->nb));
  // Plane expansions: the matrix-core front end for fp16 and bf16 x (the fp32
  // VALU one for fp32 x).  Measured on MI355X: the 70B stack at m = 8 (fp16 x)
  // 15.56 -> 15.05 ms per token.  SDQ_PLANES_MFMA=0 forces the VALU kernels
  // (a test aid, read on every launch).
  const char* pm_env = std::getenv("SDQ_PLANES_MFMA");
  const bool planes_mfma = xt != SDQ_F32 && !(pm_env && std::atoi(pm_env) == 0);
  if (mfma_base3(L, m)) {
    const int steps3 = mfma_steps3(L);
    const dim3 pgrid(static_cast<unsigned>(steps3), static_cast<unsigned>(L->nb));
#define SDQ_PLANES3(BB)                                                                          \
  if (planes_mfma && xt == SDQ_BF16)                                                             \
    expand_planes_b3_mfma_kernel<BB, true><<<pgrid, dim3(kExpThreads), 0, stream>>>(             \
        x, static_cast<int>(m), npg_for(m), L->k, L->nb, L->m_up, steps3, T->et_hi, T->et_lo,      \
        T->e1max, reinterpret_cast<uint8_t*>(w.planes), w.sx, z);                                \
  else if (planes_mfma)                                                                          \
    expand_planes_b3_mfma_kernel<BB, false><<<pgrid, dim3(kExpThreads), 0, stream>>>(            \
        x, static_cast<int>(m), npg_for(m), L->k, L->nb, L->m_up, steps3, T->et_hi, T->et_lo,      \
        T->e1max, reinterpret_cast<uint8_t*>(w.planes), w.sx, z);                                \
  else                                                                                           \
    expand_planes_b3_kernel<BB><<<pgrid, dim3(kExpThreads), 0, stream>>>(                        \
        x, xt, static_cast<int>(m), npg_for(m), L->k, L->nb, L->m_up, T->m_pad, steps3,          \
        reinterpret_cast<const float4*>(T->edec), T->e1max, reinterpret_cast<uint8_t*>(w.planes),\
        w.sx, z)
    switch (B) {
      case 64: SDQ_PLANES3(64); break;
      case 128: SDQ_PLANES3(128); break;
      default: SDQ_PLANES3(256); break;
    }
#undef SDQ_PLANES3
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_error(e, "decode expansion launch");
    return SDQ_OK;
  }
  if (use_mfma(L, m)) {
    const int npg = npg_for(m);
    const int cpb = mfma_cpb(L);
    const dim3 pgrid(static_cast<unsigned>(cpb * (L->levels == 2 ? 2 : 1)), static_cast<unsigned>(L->nb));
    // Two blocks per workgroup (E loaded once for both) for fp16 x when M is a
    // multiple of the code chunk and one block per workgroup would take
    // kPlanePairs workgroups or more (bf16 x: 248 VGPRs with two blocks).
    // Measured on MI355X at m = 8, k = 28672 (graph replay): OSR 3 16.7 ->
    // 13.0 us, OSR 2 12.2 -> 10.2 us, OSR 1.5 (672 workgroups) 9.5 -> 9.9 us.  SDQ_PLANES_NBW=1 or 2 overrides (a tuning aid,
    // read on every launch; 2 only where M allows it).
    const int64_t cpc = L->levels == 2 ? 128 : 64;
    const char* nbw_env = std::getenv("SDQ_PLANES_NBW");
    int pnb = xt == SDQ_F16 && L->m_up % cpc == 0 && static_cast<int64_t>(pgrid.x) * L->nb >= kPlanePairs ? 2 : 1;
    if (nbw_env && (std::atoi(nbw_env) == 1 || std::atoi(nbw_env) == 2)) pnb = std::atoi(nbw_env);
    if (L->m_up % cpc != 0) pnb = 1;
    const dim3 pgrid2(pgrid.x, static_cast<unsigned>((L->nb + 1) / 2));
    // One activation row: the fp32 VALU front end (the matrix-core one would
    // leave 15 of its 16 operand rows empty), two blocks per workgroup sharing
    // E when M is a multiple of the chunk and the launch has kExpRowPairs
    // (segment, block) pairs or more (SDQ_EXP_NBW=1 or 2 overrides).
    static const char* rnb_env = std::getenv("SDQ_EXP_NBW");
    int rnb = L->m_up % cpc == 0 && static_cast<int64_t>(pgrid.x) * L->nb >= kExpRowPairs ? 2 : 1;
    if (rnb_env && (std::atoi(rnb_env) == 1 || std::atoi(rnb_env) == 2)) rnb = std::atoi(rnb_env);
    if (L->m_up % cpc != 0) rnb = 1;
#define SDQ_PLANES_M(BB, LV, BF)                                                                 \
  if (pnb == 2)                                                                                  \
    expand_planes_mfma_kernel<BB, LV, BF, 2><<<pgrid2, dim3(kExpThreads), 0, stream>>>(          \
        x, static_cast<int>(m), npg, L->k, L->nb, L->m_up, cpb, T->et_hi, T->et_lo, T->e1max,      \
        w.planes, w.sx, z);                                                                      \
  else                                                                                           \
    expand_planes_mfma_kernel<BB, LV, BF, 1><<<pgrid, dim3(kExpThreads), 0, stream>>>(           \
        x, static_cast<int>(m), npg, L->k, L->nb, L->m_up, cpb, T->et_hi, T->et_lo, T->e1max,      \
        w.planes, w.sx, z)
#define SDQ_PLANES_V(BB, LV, NB_, GRID)                                                          \
  expand_planes_kernel<BB, LV, NB_><<<GRID, dim3(kExpThreads), 0, stream>>>(                     \
      x, xt, static_cast<int>(m), npg, L->k, L->nb, L->m_up, T->m_pad, cpb,                      \
      reinterpret_cast<const float4*>(T->edec), T->e1max, w.planes, w.sx, z)
#define SDQ_PLANES(BB, LV)                                                                       \
  if (m == 1 && rnb == 2) {                                                                      \
    SDQ_PLANES_V(BB, LV, 2, pgrid2);                                                             \
  } else if (m == 1) {                                                                           \
    SDQ_PLANES_V(BB, LV, 1, pgrid);                                                              \
  } else if (planes_mfma && xt == SDQ_BF16) {                                                    \
    SDQ_PLANES_M(BB, LV, true);                                                                  \
  } else if (planes_mfma) {                                                                      \
    SDQ_PLANES_M(BB, LV, false);                                                                 \
  } else                                                                                         \
    SDQ_PLANES_V(BB, LV, 1, pgrid)
    if (L->levels == 2) {
      switch (B) {
        case 64: SDQ_PLANES(64, 2); break;
        case 128: SDQ_PLANES(128, 2); break;
        default: SDQ_PLANES(256, 2); break;
      }
    } else {
      switch (B) {
        case 64: SDQ_PLANES(64, 3); break;
        case 128: SDQ_PLANES(128, 3); break;
        default: SDQ_PLANES(256, 3); break;
      }
    }
#undef SDQ_PLANES
#undef SDQ_PLANES_V
#undef SDQ_PLANES_M
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_error(e, "decode expansion launch");
    return SDQ_OK;
  }
  if (m == 1) {
    // Blocks per workgroup: two once the launch has kExpRowPairs (64-sample
    // tile, block) pairs or more, else one.  Measured on MI355X at m = 1:
    // k = 28672 at OSR 3 (1344 pairs) 5.4 -> 4.4 us with two, no gain at
    // k = 8192 (384 pairs) or k = 28672 at OSR 1.5 (672 pairs), and slower
    // with four or eight (their blocks' products run one after another).
    // SDQ_EXP_NBW=1 or 2 overrides (a tuning aid).
    static const char* env = std::getenv("SDQ_EXP_NBW");
    const int64_t tiles = T->m_pad / 64;
    int nbw = tiles * L->nb >= kExpRowPairs ? 2 : 1;
    if (env && (std::atoi(env) == 1 || std::atoi(env) == 2)) nbw = std::atoi(env);
    const dim3 rgrid(static_cast<unsigned>(tiles), static_cast<unsigned>((L->nb + nbw - 1) / nbw));
#define SDQ_ROW(BB, NBW_)                                                                       \
  expand_decode_row_kernel<BB, NBW_><<<rgrid, dim3(kExpThreads), 0, stream>>>(                  \
      x, xt, static_cast<int>(L->nb), L->m_up, T->m_pad, L->k_up, k_up_pad,                      \
      reinterpret_cast<const float4*>(T->edec), w.xt, z)
#define SDQ_ROW_B(BB)                                                                           \
  if (nbw == 2) SDQ_ROW(BB, 2);                                                                 \
  else SDQ_ROW(BB, 1)
    switch (B) {
      case 64: SDQ_ROW_B(64); break;
      case 128: SDQ_ROW_B(128); break;
      default: SDQ_ROW_B(256); break;
    }
#undef SDQ_ROW_B
#undef SDQ_ROW
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_error(e, "decode expansion launch");
    return SDQ_OK;
  }
#define SDQ_EXPAND(BB)                                                                          \
  expand_decode_kernel<BB><<<egrid, dim3(kExpThreads), 0, stream>>>(                            \
      x, xt, static_cast<int>(m), L->k, L->m_up, T->m_pad, L->k_up, k_up_pad,                   \
      reinterpret_cast<const float4*>(T->edec), w.xt, z)
  switch (B) {
    case 64: SDQ_EXPAND(64); break;
    case 128: SDQ_EXPAND(128); break;
    default: SDQ_EXPAND(256); break;
  }
#undef SDQ_EXPAND
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "decode expansion launch");
  return SDQ_OK;
}

sdq_status launch_decode_contract(int64_t m, LinearSet S, const sdq_layout* L, bool accumulate, void* ws,
                                  bool y_ready, hipStream_t stream) {
  const DecodeWs w = carve(L, m, ws);
  if (!accumulate && !y_ready && decode_needs_zero_y(L, m, set_panels(S))) {
    for (int j = 0; j < S.count; ++j) {
      const int64_t count = m * S.n[j];
      const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 4096));
      fill_zero_kernel<<<dim3(blocks), dim3(256), 0, stream>>>(S.y[j], count);
    }
  }
  if (mfma_base3(L, m)) {
    const int64_t panels = fill_first(S, panels_of);
    const int bpw = mfma_bpw(L, m, panels);
    const int splits = mfma_splits(L, m, panels);
    const dim3 grid(static_cast<unsigned>(splits), static_cast<unsigned>(panels));
#define SDQ_B3(NPG_)                                                                                  \
  gemv_mfma_b3_kernel<NPG_><<<grid, dim3(256), 0, stream>>>(                                          \
      S, reinterpret_cast<const uint4*>(w.planes), w.sx, static_cast<int>(m), L->n_chunks, L->nb, L->m_up, \
      mfma_cpb3(L), mfma_steps3(L), bpw, splits, accumulate ? 1 : 0)
    switch (npg_for(m)) {
      case 1: SDQ_B3(1); break;
      case 2: SDQ_B3(2); break;
      case 3: SDQ_B3(3); break;
      default: SDQ_B3(4); break;
    }
#undef SDQ_B3
  } else if (L->packing == SDQ_PACK_BASE3) {
    if (!decode_reads_base3(L, m)) return set_error(SDQ_ERR_ARG, "base-3 codes need unpacking on this path");
    switch (pick_seg(L, 1, set_panels(S))) {
      case 8: launch_gemv_base3_seg<8>(w, S, L, accumulate, stream); break;
      case 4: launch_gemv_base3_seg<4>(w, S, L, accumulate, stream); break;
      default: launch_gemv_base3_seg<2>(w, S, L, accumulate, stream); break;
    }
  } else if (use_mfma(L, m)) {
    if (L->levels == 2) launch_mfma_levels<2>(w, S, L, m, accumulate, stream);
    else launch_mfma_levels<3>(w, S, L, m, accumulate, stream);
  } else if (L->levels == 2) {
    launch_gemv<2>(w, S, L, m, accumulate, stream);
  } else {
    launch_gemv<3>(w, S, L, m, accumulate, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "decode GEMV launch");
  return SDQ_OK;
}

}  // namespace sdq
