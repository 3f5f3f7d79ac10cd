// Decode path of sdq_linear (m <= 16 activation rows), two launches:
//
//   expand   x_tilde = per block (x_b Had) D^T in fp32: load the block of every
//            activation row, FWHT in LDS, scale by 1/sqrt(B), then each output
//            sample o is a 256-term dot product with row o of the decimation
//            matrix D (four lanes per sample, reduced with shuffles).  Also
//            zeroes the split-K counters used by the GEMV.
//   gemv     y[i, r] = s_r * sum_j C[r, j] x_tilde[i, j] with additions only:
//            a workgroup owns one 64-row panel and one K segment; it builds, for
//            every activation row, lookup tables holding the 16 signed partial
//            sums of each 4-bit group of codes (4 binary codes or 2 ternary
//            codes), then each lane (= one weight row) streams its 16-byte code
//            chunks (one coalesced 1 KB load per wave) and adds one table entry
//            per 4 bits.  Segments of one panel are combined deterministically:
//            each writes its partial sums, and the last segment to finish
//            (a device-scope counter) adds them in segment order and applies
//            the row scale.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <hip/hip_bf16.h>

#include "sdq_internal.h"

namespace sdq {
namespace {

constexpr int kExpThreads = 256;
constexpr int kExpSlice = 64;       // output samples per expand workgroup
constexpr int kGemvWaves = 4;
constexpr int kGroupsPerChunk = 32; // 128 bits / 4

template <int MR>
struct DecodeCfg {
  static constexpr int kSegChunks = MR <= 2 ? 8 : 16 / MR;   // tables <= 32 KB
  static constexpr int kGroups = kSegChunks * kGroupsPerChunk;
  static constexpr int kLutFloats = MR * kGroups * 16;
};

__device__ inline float load_x(const void* x, sdq_dtype xt, int64_t idx) {
  if (xt == SDQ_F16) return __half2float(static_cast<const __half*>(x)[idx]);
  if (xt == SDQ_BF16) return __bfloat162float(static_cast<const __hip_bfloat16*>(x)[idx]);
  return static_cast<const float*>(x)[idx];
}

template <int B>
__global__ __launch_bounds__(kExpThreads) void expand_decode_kernel(
    const void* __restrict__ x, sdq_dtype xt, int m, int64_t k, int m_up, int64_t k_up,
    int64_t k_up_pad, float inv_sqrt_b, const float* __restrict__ dmat, float* __restrict__ xt_out,
    uint32_t* __restrict__ counters, int64_t n_counters) {
  __shared__ float h[16][B];
  const int tid = threadIdx.x;
  const int64_t b = blockIdx.x;
  const int slice = blockIdx.y;
  if (b == 0 && slice == 0) {
    for (int64_t i = tid; i < n_counters; i += kExpThreads) counters[i] = 0u;
    const int64_t pad = k_up_pad - k_up;
    for (int64_t i = tid; i < m * pad; i += kExpThreads)
      xt_out[(i / pad) * k_up_pad + k_up + (i % pad)] = 0.0f;
  }
  for (int idx = tid; idx < m * B; idx += kExpThreads) {
    const int i = idx / B;
    const int t = idx % B;
    h[i][t] = load_x(x, xt, static_cast<int64_t>(i) * k + b * B + t);
  }
  __syncthreads();
  for (int hs = 1; hs < B; hs <<= 1) {
    for (int idx = tid; idx < m * (B / 2); idx += kExpThreads) {
      const int i = idx / (B / 2);
      const int pr = idx % (B / 2);
      const int j = (pr / hs) * (2 * hs) + (pr % hs);
      const float a = h[i][j];
      const float c = h[i][j + hs];
      h[i][j] = a + c;
      h[i][j + hs] = a - c;
    }
    __syncthreads();
  }
  const int o = slice * kExpSlice + tid / 4;
  const int part = tid % 4;
  constexpr int TP = B / 4;
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  if (o < m_up) {
    const float* drow = dmat + static_cast<int64_t>(o) * B + part * TP;
    for (int t4 = 0; t4 < TP; t4 += 4) {
      const float4 d = *reinterpret_cast<const float4*>(drow + t4);
      const int t = part * TP + t4;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (i < m) {
          acc[i] += d.x * h[i][t] + d.y * h[i][t + 1] + d.z * h[i][t + 2] + d.w * h[i][t + 3];
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    float vsum = acc[i];
    vsum += __shfl_xor(vsum, 1);
    vsum += __shfl_xor(vsum, 2);
    acc[i] = vsum;
  }
  if (o < m_up && part == 0) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (i < m) xt_out[static_cast<int64_t>(i) * k_up_pad + b * m_up + o] = acc[i] * inv_sqrt_b;
  }
}

// Table entry e of a 4-bit group: binary bits b0..b3 select +x or -x for four
// consecutive samples; ternary fields f0 = e & 3, f1 = e >> 2 weight two
// samples by {00: 0, 01: +1, 11: -1, 10: 0}.
template <int LEVELS>
__device__ inline void build_group(const float* xs, float* out16) {
  if (LEVELS == 2) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float s = 0.0f;
#pragma unroll
      for (int q = 0; q < 4; ++q) s += ((e >> q) & 1) ? xs[q] : -xs[q];
      out16[e] = s;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int f0 = e & 3, f1 = e >> 2;
      const float a = f0 == 1 ? xs[0] : (f0 == 3 ? -xs[0] : 0.0f);
      const float c = f1 == 1 ? xs[1] : (f1 == 3 ? -xs[1] : 0.0f);
      out16[e] = a + c;
    }
  }
}

template <int MR, int LEVELS>
__global__ __launch_bounds__(64 * kGemvWaves) void gemv_lut_kernel(
    const uint4* __restrict__ codes, const float* __restrict__ scales,
    const float* __restrict__ xt, int m, int64_t n, int64_t n_chunks, int64_t k_up_pad,
    int n_segs, float* __restrict__ partials, uint32_t* __restrict__ counters,
    float* __restrict__ y) {
  using Cfg = DecodeCfg<MR>;
  constexpr int CPG = LEVELS == 2 ? 4 : 2;      // codes per 4-bit group
  extern __shared__ float smem[];
  float* lut = smem;                                  // [MR][kGroups][16]
  float* red = smem;                                  // [waves][MR][64], reuses the tables
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  const int64_t panel = blockIdx.x;
  const int seg = blockIdx.y;
  const int64_t c0 = static_cast<int64_t>(seg) * Cfg::kSegChunks;
  const int nch = static_cast<int>(min<int64_t>(Cfg::kSegChunks, n_chunks - c0));
  const int64_t code0 = c0 * kGroupsPerChunk * CPG;   // first code of the segment

  // Build the tables: one (activation row, group) per thread iteration.
  for (int idx = tid; idx < MR * Cfg::kGroups; idx += 64 * kGemvWaves) {
    const int i = idx / Cfg::kGroups;
    const int g = idx % Cfg::kGroups;
    float xs[CPG];
    const bool ok = i < m && g < nch * kGroupsPerChunk;
#pragma unroll
    for (int q = 0; q < CPG; ++q)
      xs[q] = ok ? xt[static_cast<int64_t>(i) * k_up_pad + code0 + g * CPG + q] : 0.0f;
    float e16[16];
    build_group<LEVELS>(xs, e16);
    float4* dst = reinterpret_cast<float4*>(lut + (static_cast<int64_t>(i) * Cfg::kGroups + g) * 16);
    dst[0] = make_float4(e16[0], e16[1], e16[2], e16[3]);
    dst[1] = make_float4(e16[4], e16[5], e16[6], e16[7]);
    dst[2] = make_float4(e16[8], e16[9], e16[10], e16[11]);
    dst[3] = make_float4(e16[12], e16[13], e16[14], e16[15]);
  }
  __syncthreads();

  float acc[MR];
#pragma unroll
  for (int i = 0; i < MR; ++i) acc[i] = 0.0f;
  const uint4* src = codes + (panel * n_chunks + c0) * kPanel + lane;
  for (int cc = wave; cc < nch; cc += kGemvWaves) {
    const uint4 q = src[static_cast<int64_t>(cc) * kPanel];
    const uint32_t words[4] = {q.x, q.y, q.z, q.w};
    const float* lbase = lut + cc * kGroupsPerChunk * 16;
#pragma unroll
    for (int wi = 0; wi < 4; ++wi) {
#pragma unroll
      for (int nib = 0; nib < 8; ++nib) {
        const uint32_t e = (words[wi] >> (4 * nib)) & 15u;
        const float* ent = lbase + (wi * 8 + nib) * 16 + e;
#pragma unroll
        for (int i = 0; i < MR; ++i) acc[i] += ent[i * Cfg::kGroups * 16];
      }
    }
  }
  // Combine the waves of this workgroup (the tables are dead from here on).
  __syncthreads();
#pragma unroll
  for (int i = 0; i < MR; ++i) red[(wave * MR + i) * 64 + lane] = acc[i];
  __syncthreads();
  const int64_t r = panel * kPanel + lane;
  if (n_segs == 1) {
    if (wave == 0 && r < n) {
      const float s = scales[r];
      for (int i = 0; i < m; ++i) {
        float tot = 0.0f;
#pragma unroll
        for (int w = 0; w < kGemvWaves; ++w) tot += red[(w * MR + i) * 64 + lane];
        y[static_cast<int64_t>(i) * n + r] = tot * s;
      }
    }
    return;
  }
  float* mypart = partials + ((panel * n_segs + seg) * MR) * 64;
  if (wave == 0) {
    for (int i = 0; i < m; ++i) {
      float tot = 0.0f;
#pragma unroll
      for (int w = 0; w < kGemvWaves; ++w) tot += red[(w * MR + i) * 64 + lane];
      mypart[i * 64 + lane] = tot;
    }
    __threadfence();
  }
  __syncthreads();
  if (tid == 0) {
    const uint32_t prev = atomicAdd(&counters[panel], 1u);
    s_last = prev == static_cast<uint32_t>(n_segs - 1);
  }
  __syncthreads();
  if (!s_last || wave != 0) return;
  __threadfence();
  if (r >= n) return;
  const float s = scales[r];
  const float* pp = partials + (panel * n_segs * MR) * 64;
  for (int i = 0; i < m; ++i) {
    float tot = 0.0f;
    for (int sg = 0; sg < n_segs; ++sg)
      tot += __hip_atomic_load(pp + (static_cast<int64_t>(sg) * MR + i) * 64 + lane,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    y[static_cast<int64_t>(i) * n + r] = tot * s;
  }
}

int round_mr(int64_t m) {
  if (m <= 1) return 1;
  if (m <= 2) return 2;
  if (m <= 4) return 4;
  if (m <= 8) return 8;
  return 16;
}

template <int MR>
int segs_for(const sdq_layout* L) {
  return static_cast<int>((L->n_chunks + DecodeCfg<MR>::kSegChunks - 1) / DecodeCfg<MR>::kSegChunks);
}

int segs_for_mr(const sdq_layout* L, int mr) {
  switch (mr) {
    case 1: return segs_for<1>(L);
    case 2: return segs_for<2>(L);
    case 4: return segs_for<4>(L);
    case 8: return segs_for<8>(L);
    default: return segs_for<16>(L);
  }
}

struct DecodeWs {
  uint32_t* counters;
  float* xt;
  float* partials;
  size_t bytes;
};

DecodeWs carve(const sdq_layout* L, int64_t m, void* base) {
  const int mr = round_mr(m);
  const int64_t n_panels = L->n_pad / kPanel;
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const int n_segs = segs_for_mr(L, mr);
  char* p = static_cast<char*>(base);
  size_t off = 0;
  DecodeWs w;
  w.counters = reinterpret_cast<uint32_t*>(p ? p + off : nullptr);
  off = align_up(off + static_cast<size_t>(n_panels) * 4, 256);
  w.xt = reinterpret_cast<float*>(p ? p + off : nullptr);
  off = align_up(off + static_cast<size_t>(m) * k_up_pad * 4, 256);
  w.partials = reinterpret_cast<float*>(p ? p + off : nullptr);
  off = align_up(off + static_cast<size_t>(n_panels) * n_segs * mr * 64 * 4, 256);
  w.bytes = off;
  return w;
}

template <int MR, int LEVELS>
void launch_gemv(const DecodeWs& w, const void* codes, const float* scales, const sdq_layout* L,
                 int64_t m, float* y, hipStream_t stream) {
  using Cfg = DecodeCfg<MR>;
  const int n_segs = segs_for<MR>(L);
  const size_t shmem = static_cast<size_t>(Cfg::kLutFloats > kGemvWaves * MR * 64
                                               ? Cfg::kLutFloats : kGemvWaves * MR * 64) * sizeof(float);
  const dim3 grid(static_cast<unsigned>(L->n_pad / kPanel), static_cast<unsigned>(n_segs));
  gemv_lut_kernel<MR, LEVELS><<<grid, dim3(64 * kGemvWaves), shmem, stream>>>(
      static_cast<const uint4*>(codes), scales, w.xt, static_cast<int>(m), L->n, L->n_chunks,
      L->n_chunks * L->codes_per_chunk, n_segs, w.partials, w.counters, y);
}

template <int MR>
void launch_gemv_levels(const DecodeWs& w, const void* codes, const float* scales,
                        const sdq_layout* L, int64_t m, float* y, hipStream_t stream) {
  if (L->levels == 2) launch_gemv<MR, 2>(w, codes, scales, L, m, y, stream);
  else launch_gemv<MR, 3>(w, codes, scales, L, m, y, stream);
}

}  // namespace

size_t decode_ws_bytes(const sdq_layout* L, int64_t m) { return carve(L, m, nullptr).bytes; }

sdq_status launch_decode(const void* x, sdq_dtype xt, int64_t m, const void* codes,
                         const float* scales, const sdq_layout* L, const Tables* T, float* y,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  (void)ws_bytes;
  const DecodeWs w = carve(L, m, ws);
  const int B = L->block;
  const float inv_sqrt_b = static_cast<float>(1.0 / std::sqrt(static_cast<double>(B)));
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const dim3 egrid(static_cast<unsigned>(L->nb), static_cast<unsigned>((L->m_up + kExpSlice - 1) / kExpSlice));
  const int64_t n_panels = L->n_pad / kPanel;
#define SDQ_EXPAND(BB)                                                                         \
  expand_decode_kernel<BB><<<egrid, dim3(kExpThreads), 0, stream>>>(                           \
      x, xt, static_cast<int>(m), L->k, L->m_up, L->k_up, k_up_pad, inv_sqrt_b, T->dmat, w.xt, \
      w.counters, n_panels)
  switch (B) {
    case 64: SDQ_EXPAND(64); break;
    case 128: SDQ_EXPAND(128); break;
    default: SDQ_EXPAND(256); break;
  }
#undef SDQ_EXPAND
  switch (round_mr(m)) {
    case 1: launch_gemv_levels<1>(w, codes, scales, L, m, y, stream); break;
    case 2: launch_gemv_levels<2>(w, codes, scales, L, m, y, stream); break;
    case 4: launch_gemv_levels<4>(w, codes, scales, L, m, y, stream); break;
    case 8: launch_gemv_levels<8>(w, codes, scales, L, m, y, stream); break;
    default: launch_gemv_levels<16>(w, codes, scales, L, m, y, stream); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "decode launch");
  return SDQ_OK;
}

}  // namespace sdq
