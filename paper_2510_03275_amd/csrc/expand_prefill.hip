// Prefill path of sdq_linear (m > 16 activation rows), the expansion, on the
// fp16 matrix cores (v_mfma_f32_32x32x16_f16, fp32 accumulation):
//
//   expand   x_tilde_b = x_b E with E = Had D^T (B x M) for every block b: a
//            batched GEMM.  E is held as an fp16 pair hi + lo, so x E_hi + x E_lo
//            reproduces the fp64 product to ~2^-22 relative for fp16 / bf16
//            inputs; fp32 inputs add x_lo E_hi.  The result is rounded once
//            to fp16 (without Had also kept as an fp16 pair, the GEMM then
//            running over both halves).
//
//   scale    fp16 holds normal numbers from 2^-14 to 65504 only, so every
//            activation row i is first multiplied by a power of two p_i
//            (exact) picked from its largest magnitude a_i:
//            a_i max(e1max, 1) p_i < 2^14.  Each x_tilde sample of the row,
//            bounded by a_i e1max, then stays below 2^14 (no overflow in x,
//            x_lo or x_tilde), and the row's large samples sit far above the
//            subnormals whatever the row's magnitude.  The GEMM multiplies
//            its sums by 1 / p_i (exact).
//
// Built with the matrix-core accumulators in VGPRs (the build sets the
// compiler's MFMA VGPR form for this file): left to its heuristics the
// compiler runs the MFMAs on AGPR copies of accumulators it carries through
// the t loop in VGPRs.
//
// MFMA operand convention: lane l supplies row (A) or column (B) l % 32 and
// the eight consecutive k of group l / 32; accumulator v holds row
// 8*(v/4) + 4*(l/32) + v%4, column l%32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <string>
#include <type_traits>
#include <hip/hip_fp16.h>
#include <hip/hip_bf16.h>

#include "sdq_internal.h"

namespace sdq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ inline floatx16 mfma32(const half8& a, const half8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Workgroups are dealt to the eight XCDs round-robin by index, and each XCD
// has its own L2.  Map workgroup `id` of `n` to a tile so that every XCD
// receives one contiguous range of tile indices (tiles that share operands
// are then numbered next to each other).
constexpr int kXcds = 8;
__device__ inline int64_t xcd_tile(int64_t id, int64_t n) {
  const int64_t xcd = id % kXcds, j = id / kXcds;
  const int64_t per = n / kXcds, rem = n % kXcds;
  return xcd * per + (xcd < rem ? xcd : rem) + j;
}

// Row factors: wave w of workgroup g takes activation row 4 g + w, reduces
// max |x| over its k values (16-byte loads, 1 KB per wave load) and writes
// p = 2^e and 1 / p with e = 14 - ceil2(a max(e1max, 1)), where ceil2(v) is
// the exponent ex of v = f 2^ex, f in [0.5, 1) (so v < 2^ex).  A row of zeros
// or with a non-finite maximum keeps p = 1.
template <sdq_dtype XT>
__global__ __launch_bounds__(256) void prefill_row_scale_kernel(const void* __restrict__ x, int64_t m,
                                                                int64_t k, float e1, float* __restrict__ fac,
                                                                _Float16* __restrict__ pad_out, int64_t k_up,
                                                                int64_t k_up_pad) {
  const int lane = threadIdx.x % 64;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + threadIdx.x / 64;
  if (i >= m) return;
  if (pad_out)   // the padding columns of this row of x_tilde
    for (int64_t j = k_up + lane; j < k_up_pad; j += 64) pad_out[i * k_up_pad + j] = static_cast<_Float16>(0.0f);
  constexpr int PER = XT == SDQ_F32 ? 4 : 8;          // values per 16 bytes
  const uint4* row = reinterpret_cast<const uint4*>(static_cast<const char*>(x) +
                                                    i * k * (XT == SDQ_F32 ? 4 : 2));
  float a = 0.0f;
  for (int64_t j = lane; j < k / PER; j += 64) {
    const uint4 u = row[j];
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (XT == SDQ_F32) {
        a = fmaxf(a, fabsf(__uint_as_float(w[q])));
      } else if (XT == SDQ_BF16) {
        a = fmaxf(a, fabsf(__uint_as_float(w[q] << 16)));
        a = fmaxf(a, fabsf(__uint_as_float(w[q] & 0xFFFF0000u)));
      } else {
        _Float16 h[2];
        __builtin_memcpy(h, &w[q], 4);
        a = fmaxf(a, fabsf(static_cast<float>(h[0])));
        a = fmaxf(a, fabsf(static_cast<float>(h[1])));
      }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off /= 2) a = fmaxf(a, __shfl_xor(a, off, 64));
  if (lane == 0) {
    const float v = a * fmaxf(e1, 1.0f);
    int e = 0;
    if (v > 0.0f && v <= 3.4e38f) {
      int ex;
      frexpf(v, &ex);
      e = min(max(14 - ex, -126), 126);
    }
    fac[i] = ldexpf(1.0f, e);
    fac[m + i] = ldexpf(1.0f, -e);
  }
}

// Tiled expansion: workgroup tile kXTM activation rows x 128 samples of one
// block, t in steps of 64 through LDS (x as fp16 hi (+ lo for fp32 inputs),
// E^T as fp16 hi and lo), so each operand element fetched from memory feeds
// many MFMA products.  The four waves form a 2 x 2 grid: wave (wr, wc) owns
// rows kXTM/2 * wr .. and samples 64 wc .. 64 wc + 63 (RT x 2 accumulator
// tiles of 32 x 32), which balances its A and B fragment reads from LDS.  LDS
// rows are padded to 72 halves: fragment reads of 16 consecutive rows fall on
// distinct banks.
constexpr int kXTN = 128, kXTK = 64, kXLd = kXTK + 8;

template <sdq_dtype XT, int kXTM>
__global__ __launch_bounds__(256) void expand_prefill_tiled_kernel(
    const void* __restrict__ x, const float* __restrict__ fac, int64_t m, int64_t k, int B, int m_up,
    int64_t k_up, int64_t k_up_pad, const uint16_t* __restrict__ et_hi,
    const uint16_t* __restrict__ et_lo, _Float16* __restrict__ xt_out,
    _Float16* __restrict__ xt_lo_out) {
  constexpr bool NEED_LO = XT == SDQ_F32;
  __shared__ __attribute__((aligned(16))) _Float16 xs[NEED_LO ? 2 : 1][kXTM * kXLd];
  __shared__ __attribute__((aligned(16))) _Float16 es[2][kXTN * kXLd];
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  // Tile order: sample tiles fastest (they share the x tile), then row tiles,
  // then blocks; dealt to the XCDs in contiguous ranges.
  const int n_st = (m_up + kXTN - 1) / kXTN;
  const int64_t n_rt = (m + kXTM - 1) / kXTM;
  const int64_t tile = xcd_tile(blockIdx.x, static_cast<int64_t>(gridDim.x));
  const int st = static_cast<int>(tile % n_st);
  const int64_t i0 = ((tile / n_st) % n_rt) * kXTM;
  const int64_t b = tile / (n_st * n_rt);
  const int c0 = st * kXTN;                         // first sample of the tile
  if (b == 0 && st == 0) {
    const int64_t pad = k_up_pad - k_up;            // zero the padding columns of these rows
    for (int64_t idx = tid; idx < kXTM * pad; idx += 256) {
      const int64_t i = i0 + idx / pad;
      if (i < m) {
        xt_out[i * k_up_pad + k_up + idx % pad] = static_cast<_Float16>(0.0f);
        if (xt_lo_out) xt_lo_out[i * k_up_pad + k_up + idx % pad] = static_cast<_Float16>(0.0f);
      }
    }
  }
  constexpr int RT = kXTM / 64;                    // 32-row tiles per wave
  constexpr int XIT = kXTM * 8 / 256;               // x loads per thread per t tile
  const int wr = wave / 2, wc = wave % 2;
  floatx16 acc[RT][2];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[rt][ct][v] = 0.0f;
  const int kg = (lane / 32) * 8;
  // Registers staging the next t tile, raw: x (kXTM rows x 64 t, eight threads
  // per row, 8 values each; rows past m load row m - 1 and are zeroed when
  // stored) and E^T (128 samples x 64 t, hi and lo; samples past M load
  // sample M - 1 and are zeroed).  All loads are unconditional, so they are
  // in flight together; conversion happens when the tile is stored to LDS.
  constexpr int XW = XT == SDQ_F32 ? 2 : 1;          // uint4 per 8 values
  uint4 xr[XIT][XW], eh[4], el[4];
  float px[XIT];                                     // p_i of the rows this thread stages
#pragma unroll
  for (int it = 0; it < XIT; ++it) px[it] = fac[min<int64_t>(i0 + (tid + 256 * it) / 8, m - 1)];
#define SDQ_FETCH(T0)                                                                          \
  do {                                                                                         \
    _Pragma("unroll") for (int it = 0; it < XIT; ++it) {                                       \
      const int idx_ = tid + 256 * it;                                                         \
      const int64_t row_ = min<int64_t>(i0 + idx_ / 8, m - 1);                                 \
      const int64_t e_ = row_ * k + b * B + (T0) + (idx_ % 8) * 8;                             \
      if (XT == SDQ_F32) {                                                                     \
        const uint4* p_ = reinterpret_cast<const uint4*>(static_cast<const float*>(x) + e_);   \
        xr[it][0] = p_[0];                                                                     \
        xr[it][XW - 1] = p_[1];                                                                \
      } else {                                                                                 \
        xr[it][0] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + e_);     \
      }                                                                                        \
    }                                                                                          \
    _Pragma("unroll") for (int it = 0; it < 4; ++it) {                                         \
      const int idx_ = tid + 256 * it;                                                         \
      const int c_ = idx_ / 8;                                                                 \
      const int cc_ = c0 + c_ < m_up ? c0 + c_ : m_up - 1;                                     \
      const int64_t off_ = static_cast<int64_t>(cc_) * B + (T0) + (idx_ % 8) * 8;              \
      eh[it] = *reinterpret_cast<const uint4*>(et_hi + off_);                                  \
      el[it] = *reinterpret_cast<const uint4*>(et_lo + off_);                                  \
    }                                                                                          \
  } while (0)
  SDQ_FETCH(0);
  for (int t0 = 0; t0 < B; t0 += kXTK) {
    __syncthreads();                                // previous tile's reads are done
#pragma unroll
    for (int it = 0; it < XIT; ++it) {
      const int idx = tid + 256 * it;
      const int r = idx / 8, sg = idx % 8;
      const bool ok = i0 + r < m;
      const float p = px[it];
      half8 hi, lo;
      if (XT == SDQ_F16) {
        const half8 h = *reinterpret_cast<const half8*>(&xr[it][0]);
#pragma unroll
        for (int q = 0; q < 8; ++q) hi[q] = static_cast<_Float16>(static_cast<float>(h[q]) * p);
      } else if (XT == SDQ_BF16) {
        const uint32_t w[4] = {xr[it][0].x, xr[it][0].y, xr[it][0].z, xr[it][0].w};
#pragma unroll
        for (int q = 0; q < 8; ++q)
          hi[q] = static_cast<_Float16>(__uint_as_float(((w[q / 2] >> (16 * (q % 2))) & 0xFFFFu) << 16) * p);
      } else {
        const uint4 u0 = xr[it][0], u1 = xr[it][XW - 1];
        const uint32_t w[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float f = __uint_as_float(w[q]) * p;
          hi[q] = static_cast<_Float16>(f);
          lo[q] = static_cast<_Float16>(f - static_cast<float>(hi[q]));
        }
      }
      if (!ok) {
#pragma unroll
        for (int q = 0; q < 8; ++q) { hi[q] = 0; lo[q] = 0; }
      }
      *reinterpret_cast<half8*>(&xs[0][r * kXLd + sg * 8]) = hi;
      if (NEED_LO) *reinterpret_cast<half8*>(&xs[NEED_LO ? 1 : 0][r * kXLd + sg * 8]) = lo;
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int idx = tid + 256 * it;
      const int c = idx / 8, sg = idx % 8;
      const uint32_t keep = c0 + c < m_up ? ~0u : 0u;   // a mask, not a select of addresses
      const uint4 h = eh[it], l = el[it];
      *reinterpret_cast<uint4*>(&es[0][c * kXLd + sg * 8]) = make_uint4(h.x & keep, h.y & keep, h.z & keep, h.w & keep);
      *reinterpret_cast<uint4*>(&es[1][c * kXLd + sg * 8]) = make_uint4(l.x & keep, l.y & keep, l.z & keep, l.w & keep);
    }
    __syncthreads();
    if (t0 + kXTK < B) SDQ_FETCH(t0 + kXTK);        // in flight during this tile's MFMAs
#pragma unroll
    for (int kk = 0; kk < kXTK; kk += 16) {
      half8 a[RT], alo[RT], bh[2], bl[2];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int r = 32 * RT * wr + 32 * rt + lane % 32;
        a[rt] = *reinterpret_cast<const half8*>(&xs[0][r * kXLd + kk + kg]);
        if (NEED_LO) alo[rt] = *reinterpret_cast<const half8*>(&xs[NEED_LO ? 1 : 0][r * kXLd + kk + kg]);
      }
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const int c = 64 * wc + 32 * ct + lane % 32;
        bh[ct] = *reinterpret_cast<const half8*>(&es[0][c * kXLd + kk + kg]);
        bl[ct] = *reinterpret_cast<const half8*>(&es[1][c * kXLd + kk + kg]);
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) {
          acc[rt][ct] = mfma32(a[rt], bh[ct], acc[rt][ct]);
          acc[rt][ct] = mfma32(a[rt], bl[ct], acc[rt][ct]);
          if (NEED_LO) acc[rt][ct] = mfma32(alo[rt], bh[ct], acc[rt][ct]);
        }
    }
  }
#pragma unroll
  for (int ct = 0; ct < 2; ++ct) {
    const int col = c0 + 64 * wc + 32 * ct + lane % 32;
    if (col >= m_up) continue;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t i = i0 + 32 * RT * wr + 32 * rt + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
        if (i < m) {
          const _Float16 hi = static_cast<_Float16>(acc[rt][ct][v]);
          xt_out[i * k_up_pad + b * m_up + col] = hi;
          if (xt_lo_out)
            xt_lo_out[i * k_up_pad + b * m_up + col] =
                static_cast<_Float16>(acc[rt][ct][v] - static_cast<float>(hi));
        }
      }
  }
}

#undef SDQ_FETCH

// E-stationary form of the same product, for fp16 and bf16 activations with
// B = 128 or 256 and a single fp16 x_tilde (the layouts with Had): E^T is the
// same for every block, so a workgroup keeps one 128-sample slice of it in
// registers, as MFMA B fragments (each wave 32 samples x B taps, hi and lo),
// loaded once, and walks a range of (64-row tile, block) items.  Each item's
// x tile goes straight from global memory to LDS (global_load_lds, 16-byte
// groups XOR-swizzled by row as in the GEMM) in a ring of four buffers, the
// next three items' copies in flight during this item's MFMAs, with the
// tile's row factors p_i copied beside it.  The products run on the activation's own type: fp16 x
// against the fp16 pair hi + lo of E, bf16 x against a bf16 pair of E formed
// in registers (hi = bf16(E), lo = bf16(E - hi), E to ~2^-17).  E^T is the
// A operand, so a lane's accumulators hold four consecutive samples of one
// x_tilde row: the sums are multiplied by p_i in fp32, rounded once to fp16
// and stored 8 bytes at a time.  Workgroups sharing an item (the slices) are
// placed on one XCD.  Barriers are plain s_barrier with explicit counter
// waits (a __syncthreads() fence would wait for the copies in flight).
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void* est_lds_ptr;
typedef __attribute__((address_space(1))) const void* est_gbl_ptr;

__device__ inline int est_swz(int r) { return (r >> 1) & 7; }
constexpr int kEstRows = 64;          // x rows per item of the E-stationary expansion
constexpr int kEstBufs = 4;           // x tiles in its LDS ring
constexpr int kEstRsrcWord3 = 0x00020000;   // raw buffer resource, dword 3

// vmcnt(n) with lgkmcnt(0) (expcnt not waited on).
constexpr int est_wait_vm_lgkm0(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4); }

template <sdq_dtype XT, int B>
__global__ __launch_bounds__(256, 1) void expand_prefill_estat_kernel(
    const void* __restrict__ x, const float* __restrict__ fac, int64_t m, int64_t k, int m_up,
    int64_t k_up, int64_t k_up_pad, int64_t nb, int n_ss, int64_t ipg, int64_t n_items,
    const uint16_t* __restrict__ et_hi, const uint16_t* __restrict__ et_lo, _Float16* __restrict__ xt_out) {
  constexpr int G = B / 8;            // 16-byte groups per x row
  constexpr int KS = B / 16;          // 16-deep k steps
  constexpr int TR = kEstRows;        // x rows per item
  constexpr int NBUF = kEstBufs;      // ring of x tiles
  constexpr int TILE = TR * B;        // halves per x tile
  constexpr int RPC = 64 / G;         // rows per 1 KB copy
  constexpr int FC = (TR / 4) / RPC;  // copies per wave per tile (a wave fills TR / 4 rows)
  constexpr int F = FC + 1;           // copies per wave per item (x and the row factors)
  constexpr int SPI = (TR / 32) * 4;  // 8-byte stores per lane per item
  static_assert(2 * F + 3 * SPI <= 63, "vmcnt range");
  constexpr bool BF = XT == SDQ_BF16;
  typedef typename std::conditional<BF, bf16x8, half8>::type frag8;
  __shared__ __attribute__((aligned(16))) uint16_t lds[NBUF * TILE + NBUF * 4 * 2 * TR];
  float* const pvb = reinterpret_cast<float*>(lds + NBUF * TILE);   // [NBUF][wave][TR] row factors
  const int tid = threadIdx.x, lane = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);
  const int id = blockIdx.x, xcd = id % kXcds, jx = id / kXcds;
  const int s = jx % n_ss;
  const int64_t g = static_cast<int64_t>(jx / n_ss) * kXcds + xcd;
  const int64_t it_begin = g * ipg, it_end = min<int64_t>(n_items, it_begin + ipg);
  if (it_begin >= it_end) return;
  // E^T fragments of this lane's sample, k = 16 ks + 8 (lane / 32) .. + 7.
  const int col = 128 * s + 32 * wave + lane % 32;
  const bool cok = col < m_up;
  frag8 eh[KS], el[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int64_t off = static_cast<int64_t>(cok ? col : 0) * B + 16 * ks + 8 * (lane / 32);
    uint4 h = *reinterpret_cast<const uint4*>(et_hi + off);
    uint4 l = *reinterpret_cast<const uint4*>(et_lo + off);
    if (!cok) h = l = make_uint4(0u, 0u, 0u, 0u);
    const half8 hh = __builtin_bit_cast(half8, h), ll = __builtin_bit_cast(half8, l);
    if constexpr (BF) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float e = static_cast<float>(hh[q]) + static_cast<float>(ll[q]);
        const __bf16 bh = static_cast<__bf16>(e);
        eh[ks][q] = bh;
        el[ks][q] = static_cast<__bf16>(e - static_cast<float>(bh));
      }
    } else {
      eh[ks] = hh;
      el[ks] = ll;
    }
  }
  const uint16_t* __restrict__ xg = static_cast<const uint16_t*>(x);
  // Copy of item `item`'s x tile and row factors into buffer `buf`: copy j of
  // wave w writes rows TR/4 w + RPC j .. (lane l: row + l / G, slot l % G,
  // which holds group (l % G) ^ swz(row)); rows past m read row m - 1.  FC
  // copies per wave, and one more (the factors) on wave 0.
  const int nb32 = static_cast<int>(nb);   // items and blocks fit 32 bits
  auto fill = [&](int buf, int64_t item) {
    const int rt = static_cast<int>(item) / nb32, b = static_cast<int>(item) - rt * nb32;
    const int64_t i0 = static_cast<int64_t>(rt) * TR;
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int r = (TR / 4) * wave + RPC * j + lane / G;
      const int64_t row = min<int64_t>(i0 + r, m - 1);
      const uint16_t* src = xg + row * k + b * B + 8 * ((lane % G) ^ est_swz(r));
      __builtin_amdgcn_global_load_lds((est_gbl_ptr)src,
                                       (est_lds_ptr)(lds + buf * TILE + ((TR / 4) * wave + RPC * j) * B), 16, 0, 0);
    }
    const float* src = fac + min<int64_t>(i0 + lane, m - 1);   // every wave its own copy
    __builtin_amdgcn_global_load_lds((est_gbl_ptr)src, (est_lds_ptr)(pvb + (buf * 4 + wave) * TR), 4, 0, 0);
  };
  // Ring of NBUF buffers, NBUF - 1 items in flight: item it sits in buffer
  // (it - it_begin) % NBUF.  Per item: wait for its copies (every wave its
  // own, counted: the copies and stores issued after them stay in flight),
  // barrier, refill the buffer the previous item used with item it + NBUF - 1,
  // then the products and the stores.  Vector memory operations complete in
  // issue order for the counter, and the counts below leave out the
  // conditional operations (wave 0's factor copy, the padding stores), so
  // each wait covers at least the item's own copies.
  for (int p = 0; p < NBUF - 1; ++p) fill(p, min<int64_t>(it_begin + p, it_end - 1));
  for (int64_t it = it_begin; it < it_end; ++it) {
    const int64_t t = it - it_begin;
    const int cur = static_cast<int>(t % NBUF);
    if (t == 0) __builtin_amdgcn_s_waitcnt(est_wait_vm_lgkm0(2 * F));
    else if (t == 1) __builtin_amdgcn_s_waitcnt(est_wait_vm_lgkm0(2 * F + SPI));
    else if (t == 2) __builtin_amdgcn_s_waitcnt(est_wait_vm_lgkm0(2 * F + 2 * SPI));
    else __builtin_amdgcn_s_waitcnt(est_wait_vm_lgkm0(2 * F + 3 * SPI));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    fill(static_cast<int>((t + NBUF - 1) % NBUF), min<int64_t>(it + NBUF - 1, it_end - 1));
    const int rt = static_cast<int>(it) / nb32, b = static_cast<int>(it) - rt * nb32;
    const int64_t i0 = static_cast<int64_t>(rt) * TR;
    const uint16_t* abuf = lds + cur * TILE;
    float pr[TR / 32];
#pragma unroll
    for (int r = 0; r < TR / 32; ++r) pr[r] = pvb[(cur * 4 + wave) * TR + 32 * r + lane % 32];
    floatx16 acc[TR / 32];
#pragma unroll
    for (int r = 0; r < TR / 32; ++r)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[r][v] = 0.0f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int gk = 2 * ks + lane / 32;
#pragma unroll
      for (int r = 0; r < TR / 32; ++r) {
        const int row = 32 * r + lane % 32;
        const frag8 a = *reinterpret_cast<const frag8*>(abuf + row * B + 8 * (gk ^ est_swz(row)));
        if constexpr (BF) {
          acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(eh[ks], a, acc[r], 0, 0, 0);
          acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(el[ks], a, acc[r], 0, 0, 0);
        } else {
          acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_f16(eh[ks], a, acc[r], 0, 0, 0);
          acc[r] = __builtin_amdgcn_mfma_f32_32x32x16_f16(el[ks], a, acc[r], 0, 0, 0);
        }
      }
    }
    // acc[r][v] = x_tilde of row i0 + 32 r + lane % 32, sample
    // 128 s + 32 w + 8 (v / 4) + 4 (lane / 32) + v % 4: four consecutive
    // samples per 8-byte store.  Buffer stores over this row tile's rows
    // below m: a row past m, or a sample past M (offset ~0), falls outside the
    // range and is dropped, so every lane issues all SPI stores (the counts
    // above rely on it).  The padding columns are zeroed by the row-scale
    // kernel.
    const int64_t rows_here = min<int64_t>(TR, m - i0);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        xt_out + i0 * k_up_pad, static_cast<short>(0), static_cast<int>(rows_here * k_up_pad * 2), kEstRsrcWord3);
#pragma unroll
    for (int r = 0; r < TR / 32; ++r) {
      const int ri = 32 * r + lane % 32;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = 128 * s + 32 * wave + 8 * q + 4 * (lane / 32);
        typedef _Float16 half4 __attribute__((ext_vector_type(4)));
        typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
        half4 h;
#pragma unroll
        for (int u = 0; u < 4; ++u) h[u] = static_cast<_Float16>(acc[r][4 * q + u] * pr[r]);
        const uint32_t off = c < m_up ? static_cast<uint32_t>((ri * k_up_pad + b * m_up + c) * 2) : 0xFFFFFFFFu;
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, h), rs, off, 0, 0);
      }
    }
  }
  // the last copies (never read) land before the workgroup's LDS is released
  __builtin_amdgcn_s_waitcnt(0);
}

}  // namespace

// Without Had the row scales follow the weights' outliers and the layer
// output can be small next to s_r |x_tilde|: one fp16 rounding of x_tilde
// then exceeds the 1e-3 budget.  Those layouts keep x_tilde as an fp16 pair
// hi + lo and run the GEMM on both.
bool prefill_split(const sdq_layout* L) { return L->hadamard == SDQ_HAD_NONE; }

sdq_status launch_prefill_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                 const Tables* T, void* ws, hipStream_t stream) {
  _Float16* xbuf = static_cast<_Float16*>(ws);
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  float* fac = reinterpret_cast<float*>(static_cast<char*>(ws) + prefill_planes_bytes(L, m));
  const dim3 sgrid(static_cast<unsigned>((m + 3) / 4));
  _Float16* xlo = prefill_split(L)
                      ? reinterpret_cast<_Float16*>(static_cast<char*>(ws) +
                                                    align_up(static_cast<size_t>(m) * k_up_pad * 2, 256))
                      : nullptr;
  // fp16 / bf16 activations, B = 128 or 256, one fp16 x_tilde: the
  // E-stationary kernel (SDQ_PREFILL_EXPAND=tiled keeps the tiled one, a
  // tuning aid).  Workgroups: one per compute unit, spread over the 128-sample
  // slices of M; each walks an even share of the (row tile, block) items.
  static const char* env = std::getenv("SDQ_PREFILL_EXPAND");
  const bool tiled_forced = env && std::string(env) == "tiled";
  const bool estat = !tiled_forced && xt != SDQ_F32 && !xlo && (L->block == 128 || L->block == 256);
  _Float16* pad_out = estat ? xbuf : nullptr;   // the E-stationary kernel leaves the padding to this one
  if (xt == SDQ_F32)
    prefill_row_scale_kernel<SDQ_F32><<<sgrid, dim3(256), 0, stream>>>(x, m, L->k, T->e1max, fac, pad_out, L->k_up, k_up_pad);
  else if (xt == SDQ_BF16)
    prefill_row_scale_kernel<SDQ_BF16><<<sgrid, dim3(256), 0, stream>>>(x, m, L->k, T->e1max, fac, pad_out, L->k_up, k_up_pad);
  else
    prefill_row_scale_kernel<SDQ_F16><<<sgrid, dim3(256), 0, stream>>>(x, m, L->k, T->e1max, fac, pad_out, L->k_up, k_up_pad);
  if (estat) {
    const int n_ss = (L->m_up + 127) / 128;
    const int64_t n_items = ((m + kEstRows - 1) / kEstRows) * L->nb;
    const int64_t cus = device_compute_units();
    const int64_t groups = ((cus + n_ss - 1) / n_ss + kXcds - 1) / kXcds * kXcds;
    const int64_t ipg = (n_items + groups - 1) / groups;
    const dim3 egrid(static_cast<unsigned>(n_ss * groups));
#define SDQ_EST(XT, BB)                                                                          \
  expand_prefill_estat_kernel<XT, BB><<<egrid, dim3(256), 0, stream>>>(                           \
      x, fac, m, L->k, L->m_up, L->k_up, k_up_pad, L->nb, n_ss, ipg, n_items, T->et_hi, T->et_lo, xbuf)
    if (xt == SDQ_BF16) {
      if (L->block == 256) SDQ_EST(SDQ_BF16, 256);
      else SDQ_EST(SDQ_BF16, 128);
    } else {
      if (L->block == 256) SDQ_EST(SDQ_F16, 256);
      else SDQ_EST(SDQ_F16, 128);
    }
#undef SDQ_EST
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_error(e, "prefill expansion launch");
    return SDQ_OK;
  }
  // Sample tiles fastest: neighbouring workgroups share the x tile.  B is a
  // multiple of the 64-wide t step for every supported block.
  constexpr int tm = 128;
  const dim3 tgrid(static_cast<unsigned>(((L->m_up + kXTN - 1) / kXTN) * L->nb * ((m + tm - 1) / tm)));
#define SDQ_XT(XT)                                                                              \
  expand_prefill_tiled_kernel<XT, tm><<<tgrid, dim3(256), 0, stream>>>(                         \
      x, fac, m, L->k, L->block, L->m_up, L->k_up, k_up_pad, T->et_hi, T->et_lo, xbuf, xlo)
  if (xt == SDQ_F32) SDQ_XT(SDQ_F32);
  else if (xt == SDQ_BF16) SDQ_XT(SDQ_BF16);
  else SDQ_XT(SDQ_F16);
#undef SDQ_XT
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "prefill expansion launch");
  return SDQ_OK;
}

}  // namespace sdq
