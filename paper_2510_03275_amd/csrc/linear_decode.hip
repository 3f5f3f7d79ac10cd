// Decode path of sdq_linear (m <= 16 activation rows), two launches:
//
//   expand   x_tilde_b = x_b E for every block b, E = Had D^T (B x M, fp32; D is
//            the Resample back to B).  A workgroup owns 64 output samples of
//            one block (one wave per quarter of t, E held in registers) and
//            all activation rows.  The workgroups also zero y when the GEMV
//            will split K.
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
constexpr int kMaxDecodeRows = 16;  // activation rows of the decode path
constexpr int kGemvWaves = 4;
constexpr int kGroupsPerChunk = 32; // 128 bits / 4

__device__ inline float load_x(const void* x, sdq_dtype xt, int64_t idx) {
  if (xt == SDQ_F16) return __half2float(static_cast<const __half*>(x)[idx]);
  if (xt == SDQ_BF16) return __bfloat162float(static_cast<const __hip_bfloat16*>(x)[idx]);
  return static_cast<const float*>(x)[idx];
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
    float* __restrict__ y_zero, int64_t y_count) {
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
  if (y_zero)
    for (int64_t i = wg * kExpThreads + tid; i < y_count; i += n_wg * kExpThreads) y_zero[i] = 0.0f;
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

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = 0.0f;
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
    const uint4* __restrict__ codes, const float* __restrict__ scales,
    const float* __restrict__ xt, int m, int64_t n, int64_t n_panels, int64_t n_chunks,
    int64_t k_up_pad, int n_segs, int accumulate, float* __restrict__ y) {
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
  const int64_t panel = static_cast<int64_t>(blockIdx.x) * kGemvWaves + wave;
  const bool panel_ok = panel < n_panels;
  const int seg = blockIdx.y;
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
    for (int j = 0; j < SEG; ++j) q[j] = src[static_cast<int64_t>(min(j, nch - 1)) * kPanel];
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
#pragma unroll
      for (int nib = 0; nib < 8; ++nib) {
        // byte offset of entry e = nibble value: 4 * e
        const uint32_t off = nib == 0 ? (words[wi] << 2) & 60u : (words[wi] >> (4 * nib - 2)) & 60u;
#pragma unroll
        for (int i = 0; i < MR; ++i)
          acc[i] += *reinterpret_cast<const float*>(lbytes + (i * kRowFloats + (c * kGroupsPerChunk + wi * 8 + nib) * 16) * 4 + off);
      }
      // With several activation rows, make each word's sums complete before
      // the next word's table reads (otherwise the compiler sinks the adds
      // and keeps every read live: register pressure).
      if (MR > 1) {
#pragma unroll
        for (int i = 0; i < MR; ++i) asm volatile("" : "+v"(acc[i]));
      }
    }
  }

  // 4. Scale and write: a plain store (or add) when the segment is the whole
  //    row, otherwise an atomic add into y (zeroed beforehand, or holding the
  //    values to accumulate onto).
  const int64_t r = panel * kPanel + lane;
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

int round_mr(int64_t m) {
  if (m <= 1) return 1;
  if (m <= 2) return 2;
  if (m <= 4) return 4;
  if (m <= 8) return 8;
  return 16;
}

// Chunks per K segment.  Larger segments amortise the table build and halve
// the atomics per step up, smaller ones give more workgroups; the largest
// segment that still yields about four workgroups per CU wins (measured on
// MI355X at m = 1: 4096 x 11008 picks 2, 28672 x 8192 picks 8).  Tables of
// MR rows x SEG chunks must fit 64 KB.
int pick_seg(const sdq_layout* L, int mr) {
  static const char* env = std::getenv("SDQ_GEMV_SEG");   // tuning aid: 2, 4 or 8
  const int max_seg = mr >= 16 ? 2 : (mr >= 8 ? 4 : 8);
  if (env) {
    const int v = std::atoi(env);
    if ((v == 2 || v == 4 || v == 8) && v <= max_seg) return v;
  }
  const int64_t panel_groups = (L->n_pad / kPanel + kGemvWaves - 1) / kGemvWaves;
  for (int seg = max_seg; seg > 2; seg /= 2)
    if (panel_groups * ((L->n_chunks + seg - 1) / seg) >= 1024) return seg;
  return 2;
}

int segs_for(const sdq_layout* L, int seg) {
  return static_cast<int>((L->n_chunks + seg - 1) / seg);
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

template <int MR, int LEVELS, int SEG>
void launch_gemv_seg(const DecodeWs& w, const void* codes, const float* scales, const sdq_layout* L,
                     int64_t m, float* y, bool accumulate, hipStream_t stream) {
  const int64_t n_panels = L->n_pad / kPanel;
  const int n_segs = segs_for(L, SEG);
  const dim3 grid(static_cast<unsigned>((n_panels + kGemvWaves - 1) / kGemvWaves),
                  static_cast<unsigned>(n_segs));
  gemv_lut_kernel<MR, LEVELS, SEG><<<grid, dim3(64 * kGemvWaves), 0, stream>>>(
      static_cast<const uint4*>(codes), scales, w.xt, static_cast<int>(m), L->n, n_panels,
      L->n_chunks, L->n_chunks * L->codes_per_chunk, n_segs, accumulate ? 1 : 0, y);
}

template <int MR, int LEVELS>
void launch_gemv_mr(const DecodeWs& w, const void* codes, const float* scales, const sdq_layout* L,
                    int64_t m, float* y, bool acc, hipStream_t stream) {
  const int seg = pick_seg(L, MR);
  if constexpr (MR <= 4) {
    if (seg == 8) return launch_gemv_seg<MR, LEVELS, 8>(w, codes, scales, L, m, y, acc, stream);
  }
  if constexpr (MR <= 8) {
    if (seg == 4) return launch_gemv_seg<MR, LEVELS, 4>(w, codes, scales, L, m, y, acc, stream);
  }
  launch_gemv_seg<MR, LEVELS, 2>(w, codes, scales, L, m, y, acc, stream);
}

template <int LEVELS>
void launch_gemv(const DecodeWs& w, const void* codes, const float* scales, const sdq_layout* L,
                 int64_t m, float* y, bool acc, hipStream_t stream) {
  switch (round_mr(m)) {
    case 1: launch_gemv_mr<1, LEVELS>(w, codes, scales, L, m, y, acc, stream); break;
    case 2: launch_gemv_mr<2, LEVELS>(w, codes, scales, L, m, y, acc, stream); break;
    case 4: launch_gemv_mr<4, LEVELS>(w, codes, scales, L, m, y, acc, stream); break;
    case 8: launch_gemv_mr<8, LEVELS>(w, codes, scales, L, m, y, acc, stream); break;
    default: launch_gemv_mr<16, LEVELS>(w, codes, scales, L, m, y, acc, stream); break;
  }
}

}  // namespace

size_t decode_ws_bytes(const sdq_layout* L, int64_t m) { return carve(L, m, nullptr).bytes; }

sdq_status decode_supported(const sdq_layout* L) {
  (void)L;
  return SDQ_OK;
}

bool decode_needs_zero_y(const sdq_layout* L, int64_t m) {
  return segs_for(L, pick_seg(L, round_mr(m))) > 1;
}

sdq_status launch_decode_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                const Tables* T, void* ws, float* y_zero, hipStream_t stream) {
  const DecodeWs w = carve(L, m, ws);
  const int B = L->block;
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const int64_t y_count = y_zero ? m * L->n : 0;
  const dim3 egrid(static_cast<unsigned>(T->m_pad / 64), static_cast<unsigned>(L->nb));
#define SDQ_EXPAND(BB)                                                                          \
  expand_decode_kernel<BB><<<egrid, dim3(kExpThreads), 0, stream>>>(                            \
      x, xt, static_cast<int>(m), L->k, L->m_up, T->m_pad, L->k_up, k_up_pad,                   \
      reinterpret_cast<const float4*>(T->edec), w.xt, y_zero, y_count)
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
                                  const sdq_layout* L, float* y, bool accumulate, void* ws,
                                  bool y_ready, hipStream_t stream) {
  const DecodeWs w = carve(L, m, ws);
  if (!accumulate && !y_ready && decode_needs_zero_y(L, m)) {
    const int64_t count = m * L->n;
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 4096));
    fill_zero_kernel<<<dim3(blocks), dim3(256), 0, stream>>>(y, count);
  }
  if (L->levels == 2) launch_gemv<2>(w, codes, scales, L, m, y, accumulate, stream);
  else launch_gemv<3>(w, codes, scales, L, m, y, accumulate, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "decode GEMV launch");
  return SDQ_OK;
}

}  // namespace sdq
