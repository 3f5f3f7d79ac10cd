// Prefill path of sdq_linear (m > 16 activation rows), two launches, both on
// the fp16 matrix cores (v_mfma_f32_32x32x16_f16, fp32 accumulation):
//
//   expand   x_tilde_b = x_b E with E = Had D^T (B x M) for every block b: a
//            batched GEMM.  E is held as an fp16 pair hi + lo, so x E_hi + x E_lo
//            reproduces the fp64 product to ~2^-22 relative for fp16 / bf16
//            inputs (both exact in fp16 at these magnitudes); fp32 inputs add
//            x_lo E_hi.  The result is rounded once to fp16.
//   gemm     y[i, r] = s_r * sum_j x_tilde[i, j] C[r, j]: the codes are expanded
//            in registers to fp16 +1 / 0 / -1 and fed to the same MFMA.  This
//            is the contraction of Fig. 5 at prefill batch sizes, where it is a
//            dense GEMM over the oversampled length.
//
// MFMA operand convention used here: lane l supplies row (A) or column (B)
// l % 32 and the eight consecutive k of group l / 32.  Any fixed pairing of
// A's and B's k slots gives the same sum, so only the row/column mapping and
// the accumulator layout (row 8*(v/4) + 4*(l/32) + v%4, column l%32 for
// accumulator v) matter.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <hip/hip_bf16.h>

#include "sdq_internal.h"

namespace sdq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kExpWaves = 4;          // expand: 32 rows x (4 x 32) samples per workgroup
constexpr int kGemmBM = 128;          // activation rows per workgroup
constexpr int kGemmBN = 128;          // weight rows per workgroup

__device__ inline floatx16 mfma32(const half8& a, const half8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Loads 8 consecutive activations as fp16 hi (and lo for fp32 inputs).
__device__ inline void load_x8(const void* x, sdq_dtype xt, int64_t idx, bool ok, half8& hi, half8& lo) {
  if (!ok) {
    for (int q = 0; q < 8; ++q) { hi[q] = 0; lo[q] = 0; }
    return;
  }
  if (xt == SDQ_F16) {
    hi = *reinterpret_cast<const half8*>(static_cast<const _Float16*>(x) + idx);
    for (int q = 0; q < 8; ++q) lo[q] = 0;
  } else if (xt == SDQ_BF16) {
    const uint4 raw = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(x) + idx);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
    for (int q = 0; q < 8; ++q) {
      const uint32_t bits = ((w[q / 2] >> (16 * (q % 2))) & 0xFFFFu) << 16;
      const float f = __uint_as_float(bits);
      hi[q] = static_cast<_Float16>(f);
      lo[q] = static_cast<_Float16>(f - static_cast<float>(hi[q]));
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(x) + idx);
    const float4 c = *reinterpret_cast<const float4*>(static_cast<const float*>(x) + idx + 4);
    const float f[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
    for (int q = 0; q < 8; ++q) {
      hi[q] = static_cast<_Float16>(f[q]);
      lo[q] = static_cast<_Float16>(f[q] - static_cast<float>(hi[q]));
    }
  }
}

__global__ __launch_bounds__(64 * kExpWaves) void expand_prefill_kernel(
    const void* __restrict__ x, sdq_dtype xt, int64_t m, int64_t k, int B, int m_up,
    int64_t k_up, int64_t k_up_pad, const uint16_t* __restrict__ et_hi,
    const uint16_t* __restrict__ et_lo, _Float16* __restrict__ xt_out) {
  const int lane = threadIdx.x % 64;
  const int wave = threadIdx.x / 64;
  const int64_t b = blockIdx.x;
  const int c0 = (blockIdx.y * kExpWaves + wave) * 32;
  const int64_t i0 = static_cast<int64_t>(blockIdx.z) * 32;
  if (b == 0 && blockIdx.y == 0) {
    // Zero the padding columns of these 32 rows.
    const int64_t pad = k_up_pad - k_up;
    for (int64_t idx = threadIdx.x; idx < 32 * pad; idx += 64 * kExpWaves) {
      const int64_t i = i0 + idx / pad;
      if (i < m) xt_out[i * k_up_pad + k_up + idx % pad] = static_cast<_Float16>(0.0f);
    }
  }
  if (c0 >= m_up) return;
  const int64_t row = i0 + lane % 32;
  const int kg = (lane / 32) * 8;
  const bool row_ok = row < m;
  const bool need_lo = xt != SDQ_F16;
  floatx16 acc;
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
  const int col = c0 + lane % 32;
  for (int t0 = 0; t0 < B; t0 += 16) {
    half8 ahi, alo;
    load_x8(x, xt, row * k + b * B + t0 + kg, row_ok, ahi, alo);
    const half8 bhi = *reinterpret_cast<const half8*>(et_hi + static_cast<int64_t>(col) * B + t0 + kg);
    const half8 blo = *reinterpret_cast<const half8*>(et_lo + static_cast<int64_t>(col) * B + t0 + kg);
    acc = mfma32(ahi, bhi, acc);
    acc = mfma32(ahi, blo, acc);
    if (need_lo) acc = mfma32(alo, bhi, acc);
  }
  for (int v = 0; v < 16; ++v) {
    const int64_t i = i0 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
    if (i < m) xt_out[i * k_up_pad + b * m_up + col] = static_cast<_Float16>(acc[v]);
  }
}

// 8 codes starting at code index kk of weight row n -> fp16 +1 / 0 / -1.
template <int LEVELS>
__device__ inline half8 load_codes8(const uint32_t* __restrict__ codes, int64_t n, int64_t n_pad,
                                    int64_t n_chunks, int64_t kk) {
  constexpr int BITS = LEVELS == 2 ? 1 : 2;
  constexpr int CPC = 128 / BITS;
  constexpr int PER_WORD = 32 / BITS;
  half8 out;
  if (n >= n_pad) {
    for (int q = 0; q < 8; ++q) out[q] = 0;
    return out;
  }
  const int64_t c = kk / CPC;
  const int qpos = static_cast<int>(kk % CPC);
  const uint32_t word = codes[(((n / kPanel) * n_chunks + c) * kPanel + n % kPanel) * 4 + qpos / PER_WORD];
  const uint32_t f = word >> (BITS * (qpos % PER_WORD));
  uint16_t h[8];
  for (int q = 0; q < 8; ++q) {
    if (LEVELS == 2) {
      h[q] = ((f >> q) & 1u) ? 0x3C00u : 0xBC00u;
    } else {
      const uint32_t fld = (f >> (2 * q)) & 3u;
      h[q] = static_cast<uint16_t>(((fld & 1u) * 0x3C00u) | ((fld >> 1) << 15));
    }
  }
  for (int q = 0; q < 8; ++q) {
    _Float16 v;
    __builtin_memcpy(&v, &h[q], 2);
    out[q] = v;
  }
  return out;
}

template <int LEVELS>
__global__ __launch_bounds__(256) void gemm_prefill_kernel(
    const _Float16* __restrict__ xt, const uint32_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t m, int64_t n, int64_t n_pad, int64_t n_chunks,
    int64_t k_up_pad, float* __restrict__ y) {
  const int lane = threadIdx.x % 64;
  const int wave = threadIdx.x / 64;
  const int wm = wave / 2, wn = wave % 2;
  const int64_t i_base = static_cast<int64_t>(blockIdx.y) * kGemmBM + wm * 64;
  const int64_t n_base = static_cast<int64_t>(blockIdx.x) * kGemmBN + wn * 64;
  const int kg = (lane / 32) * 8;
  floatx16 acc[2][2];
  for (int a = 0; a < 2; ++a)
    for (int c = 0; c < 2; ++c)
      for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.0f;
  const int64_t rows[2] = {i_base + lane % 32, i_base + 32 + lane % 32};
  const int64_t cols[2] = {n_base + lane % 32, n_base + 32 + lane % 32};
  for (int64_t k0 = 0; k0 < k_up_pad; k0 += 16) {
    half8 af[2], bf[2];
    for (int a = 0; a < 2; ++a) {
      if (rows[a] < m) af[a] = *reinterpret_cast<const half8*>(xt + rows[a] * k_up_pad + k0 + kg);
      else for (int q = 0; q < 8; ++q) af[a][q] = 0;
    }
    for (int c = 0; c < 2; ++c) bf[c] = load_codes8<LEVELS>(codes, cols[c], n_pad, n_chunks, k0 + kg);
    for (int a = 0; a < 2; ++a)
      for (int c = 0; c < 2; ++c) acc[a][c] = mfma32(af[a], bf[c], acc[a][c]);
  }
  for (int c = 0; c < 2; ++c) {
    const int64_t nn = cols[c];
    if (nn >= n) continue;
    const float s = scales[nn];
    for (int a = 0; a < 2; ++a)
      for (int v = 0; v < 16; ++v) {
        const int64_t i = i_base + a * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
        if (i < m) y[i * n + nn] = acc[a][c][v] * s;
      }
  }
}

}  // namespace

size_t prefill_ws_bytes(const sdq_layout* L, int64_t m) {
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  return align_up(static_cast<size_t>(m) * k_up_pad * 2, 256);
}

sdq_status launch_prefill_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                 const Tables* T, void* ws, hipStream_t stream) {
  _Float16* xbuf = static_cast<_Float16*>(ws);
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const dim3 egrid(static_cast<unsigned>(L->nb),
                   static_cast<unsigned>((L->m_up / 32 + kExpWaves - 1) / kExpWaves),
                   static_cast<unsigned>((m + 31) / 32));
  expand_prefill_kernel<<<egrid, dim3(64 * kExpWaves), 0, stream>>>(
      x, xt, m, L->k, L->block, L->m_up, L->k_up, k_up_pad, T->et_hi, T->et_lo, xbuf);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "prefill expansion launch");
  return SDQ_OK;
}

sdq_status launch_prefill_contract(int64_t m, const void* codes, const float* scales,
                                   const sdq_layout* L, float* y, void* ws, hipStream_t stream) {
  const _Float16* xbuf = static_cast<const _Float16*>(ws);
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const dim3 ggrid(static_cast<unsigned>((L->n + kGemmBN - 1) / kGemmBN),
                   static_cast<unsigned>((m + kGemmBM - 1) / kGemmBM));
  if (L->levels == 2)
    gemm_prefill_kernel<2><<<ggrid, dim3(256), 0, stream>>>(
        xbuf, static_cast<const uint32_t*>(codes), scales, m, L->n, L->n_pad, L->n_chunks, k_up_pad, y);
  else
    gemm_prefill_kernel<3><<<ggrid, dim3(256), 0, stream>>>(
        xbuf, static_cast<const uint32_t*>(codes), scales, m, L->n, L->n_pad, L->n_chunks, k_up_pad, y);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "prefill GEMM launch");
  return SDQ_OK;
}

}  // namespace sdq
