// Decode path of sdq_linear (m <= 16 activation rows), two launches:
//
//   expand   x_tilde_b = x_b E for every block b, E = Had D^T (B x M, fp32; D is
//            the Resample back to B).  A workgroup owns 64 output samples and a
//            group of blocks: its four lanes per sample keep their quarter of
//            the sample's column of E in registers and reuse it for every block
//            and activation row of the group (partial dots reduced with
//            shuffles).  The workgroups also zero y when the GEMV will split K.
//   gemv     y[i, r] = s_r * sum_j C[r, j] x_tilde[i, j] with additions only: a
//            workgroup owns one 64-row panel and one K segment.  Each lane (one
//            weight row) first issues the loads of its 16-byte code chunks
//            (coalesced 1 KB per wave), then the workgroup builds, per
//            activation row, lookup tables of the 16 signed partial sums of
//            every 4-bit group of codes (4 binary codes or 2 ternary codes), and
//            each lane adds one table entry per 4 bits.  When K is split into
//            several segments, each segment adds its scaled partial sums into y
//            with fp32 atomics (y was zeroed by the expansion), so the result
//            can differ between runs in the last bits; a single segment stores.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <hip/hip_bf16.h>

#include <cstdio>
#include <cstdlib>
#include <algorithm>

#include "sdq_internal.h"

namespace sdq {
namespace {

constexpr int kExpThreads = 256;
constexpr int kExpSlice = 64;       // output samples per expand workgroup
constexpr int kExpBlocks = 4;       // blocks per expand workgroup (E reuse)
constexpr int kGemvWaves = 4;
constexpr int kGroupsPerChunk = 32; // 128 bits / 4

__device__ inline float load_x(const void* x, sdq_dtype xt, int64_t idx) {
  if (xt == SDQ_F16) return __half2float(static_cast<const __half*>(x)[idx]);
  if (xt == SDQ_BF16) return __bfloat162float(static_cast<const __hip_bfloat16*>(x)[idx]);
  return static_cast<const float*>(x)[idx];
}

// One workgroup: kExpSlice output samples x up to kExpBlocks blocks x all m
// rows.  The activation blocks are staged in LDS as fp32 (16 block-rows per
// pass); each lane keeps its quarter of E's column for its sample in registers.
template <int B>
__global__ __launch_bounds__(kExpThreads) void expand_decode_kernel(
    const void* __restrict__ x, sdq_dtype xt, int m, int64_t k, int64_t nb, int m_up,
    int64_t k_up, int64_t k_up_pad, const float* __restrict__ et, float* __restrict__ xt_out,
    float* __restrict__ y_zero, int64_t y_count) {
  constexpr int TP = B / 4;               // t values per lane
  constexpr int kRowsPerPass = 16;        // block-rows staged per pass
  __shared__ float xs[kRowsPerPass][B];
  const int tid = threadIdx.x;
  const int o = blockIdx.x * kExpSlice + tid / 4;
  const int part = tid % 4;
  const int64_t b0 = static_cast<int64_t>(blockIdx.y) * kExpBlocks;
  const int nbl = static_cast<int>(min<int64_t>(kExpBlocks, nb - b0));
  const int64_t wg = static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t n_wg = static_cast<int64_t>(gridDim.x) * gridDim.y;
  // The GEMV accumulates into y with atomics when it splits K: start from zero.
  if (y_zero)
    for (int64_t i = wg * kExpThreads + tid; i < y_count; i += n_wg * kExpThreads) y_zero[i] = 0.0f;
  if (wg == 0) {
    const int64_t pad = k_up_pad - k_up;
    for (int64_t i = tid; i < m * pad; i += kExpThreads)
      xt_out[(i / pad) * k_up_pad + k_up + (i % pad)] = 0.0f;
  }
  const bool live = o < m_up;
  float e[TP];
  const float* erow = et + static_cast<int64_t>(live ? o : 0) * B + part * TP;
#pragma unroll
  for (int t = 0; t < TP; t += 4) {
    const float4 v = *reinterpret_cast<const float4*>(erow + t);
    e[t] = v.x; e[t + 1] = v.y; e[t + 2] = v.z; e[t + 3] = v.w;
  }
  const int total = m * nbl;              // (row, block) pairs of this workgroup
  for (int p0 = 0; p0 < total; p0 += kRowsPerPass) {
    const int np = min(kRowsPerPass, total - p0);
    __syncthreads();
    for (int idx = tid; idx < np * B; idx += kExpThreads) {
      const int pr = idx / B, t = idx % B;
      const int i = (p0 + pr) / nbl, bb = (p0 + pr) % nbl;
      xs[pr][t] = load_x(x, xt, static_cast<int64_t>(i) * k + (b0 + bb) * B + t);
    }
    __syncthreads();
    for (int pr = 0; pr < np; ++pr) {
      const float* xr = &xs[pr][part * TP];
      float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
      for (int t = 0; t < TP; t += 4) {
        const float4 v = *reinterpret_cast<const float4*>(xr + t);
        a0 += e[t] * v.x;
        a1 += e[t + 1] * v.y;
        a2 += e[t + 2] * v.z;
        a3 += e[t + 3] * v.w;
      }
      float acc = (a0 + a1) + (a2 + a3);
      acc += __shfl_xor(acc, 1);
      acc += __shfl_xor(acc, 2);
      const int i = (p0 + pr) / nbl, bb = (p0 + pr) % nbl;
      if (live && part == 0) xt_out[static_cast<int64_t>(i) * k_up_pad + (b0 + bb) * m_up + o] = acc;
    }
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = 0.0f;
}

// Table entry e of a 4-bit group: binary bits b0..b3 select +x or -x for four
// consecutive samples; ternary fields f0 = e & 3, f1 = e >> 2 weight two
// samples by {00: 0, 01: +1, 11: -1, 10: 0}.
template <int LEVELS>
__device__ inline void build_group(const float (&xs)[4], float* out16) {
  if (LEVELS == 2) {
    const float a0 = xs[0] + xs[1], a1 = xs[0] - xs[1];
    const float c0 = xs[2] + xs[3], c1 = xs[2] - xs[3];
    const float lo[4] = {-a0, a1, -a1, a0};     // bits 1..0 = 00, 01, 10, 11
    const float hi[4] = {-c0, c1, -c1, c0};     // bits 3..2
#pragma unroll
    for (int e = 0; e < 16; ++e) out16[e] = lo[e & 3] + hi[e >> 2];
  } else {
    const float v0[4] = {0.0f, xs[0], 0.0f, -xs[0]};
    const float v1[4] = {0.0f, xs[1], 0.0f, -xs[1]};
#pragma unroll
    for (int e = 0; e < 16; ++e) out16[e] = v0[e & 3] + v1[e >> 2];
  }
}

template <int MR, int LEVELS, int SEG, int PPW>
__global__ __launch_bounds__(64 * kGemvWaves) void gemv_lut_kernel(
    const uint4* __restrict__ codes, const float* __restrict__ scales,
    const float* __restrict__ xt, int m, int64_t n, int64_t n_panels, int64_t n_chunks,
    int64_t k_up_pad, int n_segs, float* __restrict__ y) {
  constexpr int CPG = LEVELS == 2 ? 4 : 2;          // codes per 4-bit group
  constexpr int kGroups = SEG * kGroupsPerChunk;
  constexpr int NS = kGemvWaves / PPW;               // waves sharing one panel
  constexpr int kChunksPerWave = (SEG + NS - 1) / NS;
  extern __shared__ float smem[];
  float* lut = smem;                                  // [MR][kGroups][16]
  float* red = smem;                                  // [waves][MR][64], reuses the tables

  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  const int64_t panel = static_cast<int64_t>(blockIdx.x) * PPW + wave % PPW;
  const int sub = wave / PPW;
  const bool panel_ok = panel < n_panels;
  const int seg = blockIdx.y;
  const int64_t c0 = static_cast<int64_t>(seg) * SEG;
  const int nch = static_cast<int>(min<int64_t>(SEG, n_chunks - c0));
  const int64_t code0 = c0 * kGroupsPerChunk * CPG;   // first code of the segment

  // 1. Loads, in this order: the activation samples the tables need, then this
  //    lane's code chunks.  Vector memory returns in order, so the table build
  //    waits only for the former while the code stream is in flight.
  constexpr int kBuildIters = MR * kGroups / (64 * kGemvWaves);
  static_assert(kBuildIters * 64 * kGemvWaves == MR * kGroups, "one group per thread per iteration");
  float4 xv[kBuildIters];          // raw samples (only .x, .y used for ternary groups)
#pragma unroll
  for (int it = 0; it < kBuildIters; ++it) {
    const int idx = tid + it * 64 * kGemvWaves;
    const int i = idx / kGroups;
    const int g = idx % kGroups;
    const bool ok = i < m && g < nch * kGroupsPerChunk;
    const float* xp = xt + (ok ? static_cast<int64_t>(i) * k_up_pad + code0 + g * CPG : 0);
    if (CPG == 4) {
      xv[it] = *reinterpret_cast<const float4*>(xp);
    } else {
      const float2 v = *reinterpret_cast<const float2*>(xp);
      xv[it] = make_float4(v.x, v.y, 0.f, 0.f);
    }
  }
  __builtin_amdgcn_sched_barrier(0);   // keep the code loads behind the sample loads
  uint4 q[kChunksPerWave];
  const uint4* src = codes + ((panel_ok ? panel : 0) * n_chunks + c0) * kPanel + lane;
#pragma unroll
  for (int j = 0; j < kChunksPerWave; ++j) {
    // Chunks past the segment end read a valid chunk; their tables are zero.
    const int cc = min(sub + j * NS, nch - 1);
    q[j] = src[static_cast<int64_t>(cc) * kPanel];
  }
  __builtin_amdgcn_sched_barrier(0);

  // 2. Tables: 16 entries per (activation row, group); groups outside the
  //    segment or rows >= m get all-zero entries.
#pragma unroll
  for (int it = 0; it < kBuildIters; ++it) {
    const int idx = tid + it * 64 * kGemvWaves;
    const int i = idx / kGroups;
    const int g = idx % kGroups;
    const bool ok = i < m && g < nch * kGroupsPerChunk;
    const float xs[4] = {ok ? xv[it].x : 0.f, ok ? xv[it].y : 0.f, ok ? xv[it].z : 0.f,
                         ok ? xv[it].w : 0.f};
    float e16[16];
    build_group<LEVELS>(xs, e16);
    float4* dst = reinterpret_cast<float4*>(lut + static_cast<int64_t>(idx) * 16);
    dst[0] = make_float4(e16[0], e16[1], e16[2], e16[3]);
    dst[1] = make_float4(e16[4], e16[5], e16[6], e16[7]);
    dst[2] = make_float4(e16[8], e16[9], e16[10], e16[11]);
    dst[3] = make_float4(e16[12], e16[13], e16[14], e16[15]);
  }
  __syncthreads();

  // 3. Lookups: one table entry per 4 bits of code.
  float acc[MR];
#pragma unroll
  for (int i = 0; i < MR; ++i) acc[i] = 0.0f;
#pragma unroll
  for (int j = 0; j < kChunksPerWave; ++j) {
    const int cc = sub + j * NS;
    // Compile-time true unless the segment has fewer chunks than waves per panel.
    if (SEG % NS == 0 || cc < SEG) {
      const uint32_t words[4] = {q[j].x, q[j].y, q[j].z, q[j].w};
      const float* lbase = lut + cc * kGroupsPerChunk * 16;
#pragma unroll
      for (int wi = 0; wi < 4; ++wi) {
#pragma unroll
        for (int nib = 0; nib < 8; ++nib) {
          const uint32_t e = (words[wi] >> (4 * nib)) & 15u;
          const float* ent = lbase + (wi * 8 + nib) * 16 + e;
#pragma unroll
          for (int i = 0; i < MR; ++i) acc[i] += ent[i * kGroups * 16];
        }
      }
    }
  }

  // 4. Combine the waves that share a panel (the tables are dead from here on),
  //    scale, and write y: a plain store when the segment is the whole row,
  //    otherwise an atomic add into the y that the expansion zeroed.
  __syncthreads();
  if (NS > 1) {
#pragma unroll
    for (int i = 0; i < MR; ++i) red[(wave * MR + i) * 64 + lane] = acc[i];
    __syncthreads();
  }
  const int64_t r = panel * kPanel + lane;
  if (sub != 0 || !panel_ok || r >= n) return;
  const float s = scales[r];
#pragma unroll
  for (int i = 0; i < MR; ++i) {
    if (i >= m) break;
    float tot = acc[i];
    if (NS > 1) {
      tot = 0.0f;
#pragma unroll
      for (int w = 0; w < NS; ++w) tot += red[((wave + w * PPW) * MR + i) * 64 + lane];
    }
    if (n_segs == 1) y[static_cast<int64_t>(i) * n + r] = tot * s;
    else unsafeAtomicAdd(&y[static_cast<int64_t>(i) * n + r], tot * s);
  }
}

int round_mr(int64_t m) {
  if (m <= 1) return 1;
  if (m <= 2) return 2;
  if (m <= 4) return 4;
  if (m <= 8) return 8;
  return 16;
}

// Tile choice: chunks per K segment and panels per workgroup.
struct GemvTile {
  int seg;
  int ppw;
};

GemvTile pick_tile(const sdq_layout* L, int mr) {
  GemvTile t{mr <= 2 ? 8 : 16 / mr, 1};
  static const char* env = std::getenv("SDQ_GEMV_TILE");   // "seg,ppw" (tuning aid)
  if (env && mr == 1) {
    int a = 0, b = 0;
    if (std::sscanf(env, "%d,%d", &a, &b) == 2 && (a == 8 || a == 16) && (b == 1 || b == 4)) return {a, b};
  }
  // Measured on MI355X (m = 1): eight chunks per segment and one panel per
  // workgroup beat sharing tables across four panels at every layer size.
  return t;
}

int segs_for(const sdq_layout* L, const GemvTile& t) {
  return static_cast<int>((L->n_chunks + t.seg - 1) / t.seg);
}

struct DecodeWs {
  float* xt;
  size_t bytes;
};

// Workspace: x_tilde (m x k_up_pad fp32) at offset 0, so one expansion can
// serve several linears that share its (k, block, M, levels).
DecodeWs carve(const sdq_layout* L, int64_t m, void* base) {
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  DecodeWs w;
  w.xt = static_cast<float*>(base);
  w.bytes = align_up(static_cast<size_t>(m) * k_up_pad * 4, 256);
  return w;
}

template <int MR, int LEVELS, int SEG, int PPW>
void launch_gemv_tile(const DecodeWs& w, const void* codes, const float* scales, const sdq_layout* L,
                      int64_t m, float* y, hipStream_t stream) {
  constexpr int kLutFloats = MR * SEG * kGroupsPerChunk * 16;
  const int64_t n_panels = L->n_pad / kPanel;
  const int n_segs = static_cast<int>((L->n_chunks + SEG - 1) / SEG);
  const size_t shmem = static_cast<size_t>(kLutFloats > kGemvWaves * MR * 64
                                               ? kLutFloats : kGemvWaves * MR * 64) * sizeof(float);
  const dim3 grid(static_cast<unsigned>((n_panels + PPW - 1) / PPW), static_cast<unsigned>(n_segs));
  gemv_lut_kernel<MR, LEVELS, SEG, PPW><<<grid, dim3(64 * kGemvWaves), shmem, stream>>>(
      static_cast<const uint4*>(codes), scales, w.xt, static_cast<int>(m), L->n, n_panels,
      L->n_chunks, L->n_chunks * L->codes_per_chunk, n_segs, y);
}

template <int LEVELS>
void launch_gemv(const DecodeWs& w, const void* codes, const float* scales, const sdq_layout* L,
                 int64_t m, float* y, hipStream_t stream) {
  const int mr = round_mr(m);
  const GemvTile t = pick_tile(L, mr);
  switch (mr) {
    case 1:
      if (t.seg == 16 && t.ppw == 4) launch_gemv_tile<1, LEVELS, 16, 4>(w, codes, scales, L, m, y, stream);
      else if (t.seg == 16) launch_gemv_tile<1, LEVELS, 16, 1>(w, codes, scales, L, m, y, stream);
      else if (t.ppw == 4) launch_gemv_tile<1, LEVELS, 8, 4>(w, codes, scales, L, m, y, stream);
      else launch_gemv_tile<1, LEVELS, 8, 1>(w, codes, scales, L, m, y, stream);
      break;
    case 2:
      if (t.ppw == 4) launch_gemv_tile<2, LEVELS, 8, 4>(w, codes, scales, L, m, y, stream);
      else launch_gemv_tile<2, LEVELS, 8, 1>(w, codes, scales, L, m, y, stream);
      break;
    case 4: launch_gemv_tile<4, LEVELS, 4, 1>(w, codes, scales, L, m, y, stream); break;
    case 8: launch_gemv_tile<8, LEVELS, 2, 1>(w, codes, scales, L, m, y, stream); break;
    default: launch_gemv_tile<16, LEVELS, 1, 1>(w, codes, scales, L, m, y, stream); break;
  }
}

}  // namespace

size_t decode_ws_bytes(const sdq_layout* L, int64_t m) { return carve(L, m, nullptr).bytes; }

sdq_status decode_supported(const sdq_layout* L) {
  (void)L;
  return SDQ_OK;
}

bool decode_needs_zero_y(const sdq_layout* L, int64_t m) {
  return segs_for(L, pick_tile(L, round_mr(m))) > 1;
}

sdq_status launch_decode_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                const Tables* T, void* ws, float* y_zero, hipStream_t stream) {
  const DecodeWs w = carve(L, m, ws);
  const int B = L->block;
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const int64_t y_count = y_zero ? m * L->n : 0;
  const dim3 egrid(static_cast<unsigned>((L->m_up + kExpSlice - 1) / kExpSlice),
                   static_cast<unsigned>((L->nb + kExpBlocks - 1) / kExpBlocks));
#define SDQ_EXPAND(BB)                                                                        \
  expand_decode_kernel<BB><<<egrid, dim3(kExpThreads), 0, stream>>>(                          \
      x, xt, static_cast<int>(m), L->k, L->nb, L->m_up, L->k_up, k_up_pad, T->et32, w.xt,     \
      y_zero, y_count)
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

sdq_status launch_decode_contract(int64_t m, const void* codes, const float* scales,
                                  const sdq_layout* L, float* y, void* ws, bool y_zeroed,
                                  hipStream_t stream) {
  const DecodeWs w = carve(L, m, ws);
  if (!y_zeroed && decode_needs_zero_y(L, m)) {
    const int64_t count = m * L->n;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 4096));
    fill_zero_kernel<<<dim3(blocks), dim3(256), 0, stream>>>(y, count);
  }
  if (L->levels == 2) launch_gemv<2>(w, codes, scales, L, m, y, stream);
  else launch_gemv<3>(w, codes, scales, L, m, y, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "decode GEMV launch");
  return SDQ_OK;
}

}  // namespace sdq
