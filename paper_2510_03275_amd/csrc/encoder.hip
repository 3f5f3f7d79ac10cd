// Sigma-Delta weight encoder for gfx950 (Algorithm 1 without block
// compensation).  Four launches on the caller's stream:
//
//   clear      zero the non-finite flag and the per-row maxima;
//   rotate     per (64-row panel, block): load W, Sylvester FWHT in registers in
//              the stage order h = 1, 2, ..., B/2, scale by fp32(1/sqrt(B))
//              (Section 3.3), store the rotated block rows-contiguous, copy the
//              samples whose interpolation kernel is a unit impulse
//              (m % P == 0) into the upsampled buffer, fold |v| into the row max;
//   upsample   the remaining M - gcd(B, M) samples of every block as dense
//              sums x_up[m] = sum_t fl(v[t] * g(p(t, m))) in t order from +0.0,
//              every product and sum rounded separately (the Resample of
//              Algorithm 1 in closed form).  This is a batched fp32 product
//              V^T (rows x B) * U (B x M_nz) evaluated as a register-tiled VALU
//              GEMM whose k-loop runs t = 0 .. B-1 in order, so each output's
//              accumulation order is exactly the definition's;
//   scan       per (row, block) chain: first-order Sigma-Delta (Eq. 7-8) with the
//              row scale s = max|x_up| and the binary (Eq. 4) or ternary (Eq. 6,
//              threshold s/2) quantizer, packing codes into the panel format.
//
// Everything is compiled with floating-point contraction off: no fused
// multiply-add may merge a product into a sum.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <utility>

#include "sdq_internal.h"

#pragma clang fp contract(off)

namespace sdq {
namespace {

constexpr int kRotThreads = 256;
constexpr int kUpBM = 128;        // rows per upsample tile (two panels)
constexpr int kUpBN = 64;         // non-impulse samples per upsample tile
constexpr int kUpBK = 16;         // t-chunk staged in LDS (two buffers)
constexpr int kUpThreads = 128;   // 16 x 8 threads, 8 x 8 outputs each
constexpr int kScanWaves = 4;

__global__ void clear_kernel(uint32_t* __restrict__ flag, uint32_t* __restrict__ rmax, int64_t n) {
  const int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  if (i == 0) flag[0] = 0u;
  if (i < n) rmax[i] = 0u;
}

// Sign words of the signed Had (bit t set <=> s_t = -1), passed by value.
struct SignMask {
  uint32_t w[8];
};

// One workgroup: 64 rows x one block of B columns, four lanes per row.  Lane
// (row, q) holds the B/4 elements t = 16 j + 4 q + e (j < B/16, e < 4) of its
// row, loaded as float4 (a wave reads 64 contiguous bytes of each of its 16
// rows per load).  For the signed Had the signs flip first (exact); the
// transform (skipped for Had = I) runs in registers in the stage order
// h = 1, 2 (bits of e), 4, 8 (bits of q: partner lanes xor 1, 2), 16, ...,
// B/2 (bits of j); every stage pairs the same elements and rounds the same
// sums and differences as the textbook loop, so the result is bit-identical.
template <int B>
__global__ __launch_bounds__(kRotThreads) void rotate_kernel(
    const float* __restrict__ w, int64_t n, int64_t k, int64_t n_ws, int64_t k_up, int m_up,
    int g0, int phases, int had, SignMask sm, float inv_sqrt_b, float* __restrict__ v,
    float* __restrict__ xup, uint32_t* __restrict__ rmax, uint32_t* __restrict__ flag) {
  constexpr int J = B / 16;
  const int tid = threadIdx.x;
  const int q = tid & 3;
  const int rl = tid >> 2;                      // row within the panel
  const int64_t panel = blockIdx.x;
  const int64_t b = blockIdx.y;
  const int64_t r = panel * kPanel + rl;
  float x[J][4];
  bool bad = false;
  if (r < n) {
    const float4* src = reinterpret_cast<const float4*>(w + r * k + b * B) + q;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const float4 t4 = src[4 * j];
      x[j][0] = t4.x; x[j][1] = t4.y; x[j][2] = t4.z; x[j][3] = t4.w;
    }
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) bad |= !isfinite(x[j][e]);
  } else {
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[j][e] = 0.0f;   // padding rows: zeros
  }
  if (bad) atomicOr(flag, 1u);
  // Signed Had = diag(s) H / sqrt(B): flip the sign of w_t where s_t = -1
  // (exact); element (j, e) of this lane is t = 16 j + 4 q + e, in sign word
  // j / 2 at bit 16 (j % 2) + 4 q + e.
  if (had == SDQ_HAD_SIGNED) {
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t bit = (sm.w[j / 2] >> (16 * (j % 2) + 4 * q + e)) & 1u;
        x[j][e] = __uint_as_float(__float_as_uint(x[j][e]) ^ (bit << 31));
      }
  }
  // Had = I: no transform (the launch passes a scale of 1).
  if (had != SDQ_HAD_NONE) {
  // h = 1, 2: inside the float4.
#pragma unroll
  for (int j = 0; j < J; ++j) {
    float a = x[j][0], c = x[j][1];
    x[j][0] = a + c; x[j][1] = a - c;
    a = x[j][2]; c = x[j][3];
    x[j][2] = a + c; x[j][3] = a - c;
    a = x[j][0]; c = x[j][2];
    x[j][0] = a + c; x[j][2] = a - c;
    a = x[j][1]; c = x[j][3];
    x[j][1] = a + c; x[j][3] = a - c;
  }
  // h = 4, 8: across the row's four lanes (quad permutations).  The lower
  // element of a pair keeps own + partner, the upper one partner + (-own)
  // (= partner - own exactly).
#pragma unroll
  for (int bit = 1; bit <= 2; bit <<= 1) {
    const bool lower = (q & bit) == 0;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int own = __float_as_int(x[j][e]);
        // quad_perm [1,0,3,2] (xor 1) or [2,3,0,1] (xor 2)
        const float o = __int_as_float(bit == 1 ? __builtin_amdgcn_mov_dpp(own, 0xB1, 0xF, 0xF, false)
                                                : __builtin_amdgcn_mov_dpp(own, 0x4E, 0xF, 0xF, false));
        const float mine = lower ? x[j][e] : -x[j][e];
        x[j][e] = o + mine;
      }
  }
  // h = 16 .. B/2: across j, in registers.
#pragma unroll
  for (int hj = 1; hj < J; hj <<= 1)
#pragma unroll
    for (int j = 0; j < J; ++j)
      if ((j & hj) == 0)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a = x[j][e], c = x[j + hj][e];
          x[j][e] = a + c;
          x[j + hj][e] = a - c;
        }
  }
  // Scale; store rows-contiguous per t; copy the unit-impulse samples
  // (t = i * B / g0 feeds sample m = i * P); fold their |v| into the row max.
  const int stride_mask = B / g0 - 1;          // B / g0 is a power of two
  const int stride_shift = __builtin_ctz(B / g0);
  float* vq = v + (b * B + 4 * q) * n_ws + r;
  float* xq = xup + (panel * k_up + b * m_up) * kPanel + rl;
  float mx = 0.0f;
#pragma unroll
  for (int j = 0; j < J; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int t = 16 * j + 4 * q + e;
      const float val = x[j][e] * inv_sqrt_b;
      vq[static_cast<int64_t>(16 * j + e) * n_ws] = val;
      if ((t & stride_mask) == 0) {
        xq[static_cast<int64_t>((t >> stride_shift) * phases) * kPanel] = val;
        mx = fmaxf(mx, fabsf(val));
      }
    }
  mx = fmaxf(mx, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(mx), 0xB1, 0xF, 0xF, false)));
  mx = fmaxf(mx, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(mx), 0x4E, 0xF, 0xF, false)));
  if (q == 0 && r < n) atomicMax(&rmax[r], __float_as_uint(mx));
}

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) const void* gbl_void_ptr;

// Plain s_barrier between compiler fences: __syncthreads() adds a release
// fence, which would wait for the copies still in flight.
__device__ inline void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Batched VALU GEMM over (block, row tile, sample tile).  Thread (tx, ty)
// owns rows ty*8 .. ty*8+7 and tile columns tx*8 .. tx*8+7.  The t chunks
// are copied from global memory straight into two LDS buffers
// (global_load_lds_dwordx4: 1 KB per wave and copy, no staging registers);
// chunk c + 2 is copied while chunk c + 1 is multiplied.  Every output adds
// its products in increasing t, as a plain loop over t would.
__global__ __launch_bounds__(kUpThreads) void upsample_kernel(
    const float* __restrict__ v, const float* __restrict__ unz, int64_t n, int64_t n_ws,
    int64_t k_up, int B, int m_up, int phases, int m_nz, int m_nz_pad, float* __restrict__ xup,
    uint32_t* __restrict__ rmax) {
  static_assert(kUpThreads == 128 && kUpBK == 16 && kUpBM == 128 && kUpBN == 64,
                "copy pattern: each wave copies 8 of the 16 t rows of both operands");
  __shared__ __attribute__((aligned(1024))) float As0[kUpBK][kUpBM];
  __shared__ __attribute__((aligned(1024))) float As1[kUpBK][kUpBM];
  __shared__ __attribute__((aligned(1024))) float Bs0[kUpBK][kUpBN];
  __shared__ __attribute__((aligned(1024))) float Bs1[kUpBK][kUpBN];
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  const int tx = tid % 8;
  const int ty = tid / 8;
  const int64_t rt = blockIdx.x;     // row tile
  const int jt = blockIdx.y;         // sample tile
  const int64_t b = blockIdx.z;      // block
  const int64_t r0 = rt * kUpBM;
  const int j0 = jt * kUpBN;
  float acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0f;

  // Copies of one chunk by wave w: t rows 8w .. 8w+7 of A (four copies of
  // two 512-byte rows) and of B (two copies of four 256-byte rows).  Lane l
  // of a copy lands 16 l bytes past the copy's LDS base, so the global
  // source of lane l is the float4 that belongs there.
  const float* a_src = v + b * B * n_ws + (8 * wave + lane / 32) * n_ws + r0 + (lane % 32) * 4;
  const float* b_src = unz + (8 * wave + lane / 16) * m_nz_pad + j0 + (lane % 16) * 4;
#define SDQ_UP_FILL(AS, BS, C)                                                                    \
  do {                                                                                            \
    const int64_t t0_ = static_cast<int64_t>(C) * kUpBK;                                          \
    _Pragma("unroll") for (int j = 0; j < 4; ++j)                                                 \
      __builtin_amdgcn_global_load_lds((gbl_void_ptr)(a_src + (t0_ + 2 * j) * n_ws),              \
                                       (lds_void_ptr)(&AS[8 * wave + 2 * j][0]), 16, 0, 0);       \
    _Pragma("unroll") for (int j = 0; j < 2; ++j)                                                 \
      __builtin_amdgcn_global_load_lds((gbl_void_ptr)(b_src + (t0_ + 4 * j) * m_nz_pad),          \
                                       (lds_void_ptr)(&BS[8 * wave + 4 * j][0]), 16, 0, 0);       \
  } while (0)
#define SDQ_UP_MUL(AS, BS)                                                                        \
  do {                                                                                            \
    _Pragma("unroll 4") for (int tt = 0; tt < kUpBK; ++tt) {                                      \
      const float4 a0 = *reinterpret_cast<const float4*>(&AS[tt][ty * 8]);                        \
      const float4 a1 = *reinterpret_cast<const float4*>(&AS[tt][ty * 8 + 4]);                    \
      const float4 b0 = *reinterpret_cast<const float4*>(&BS[tt][tx * 8]);                        \
      const float4 b1 = *reinterpret_cast<const float4*>(&BS[tt][tx * 8 + 4]);                    \
      const float a[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};                        \
      const float c[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};                        \
      _Pragma("unroll") for (int i = 0; i < 8; ++i)                                               \
        _Pragma("unroll") for (int j = 0; j < 8; ++j) {                                           \
          const float prod = a[i] * c[j];                                                         \
          acc[i][j] = acc[i][j] + prod;                                                           \
        }                                                                                         \
    }                                                                                             \
  } while (0)

  // nc = B / 16 is even (B is 64, 128 or 256).  Chunk c + 1 is copied while
  // chunk c is multiplied; then a wait for this wave's copies (vmcnt 0) and
  // a barrier make every wave's copies visible and order the refill of a
  // buffer after every read of it.  No copy is in flight where the loop
  // closes, so the compiler can tell each buffer's reads from the other
  // buffer's copies and adds no wait of its own before them.
  const int nc = B / kUpBK;
  SDQ_UP_FILL(As0, Bs0, 0);
  __builtin_amdgcn_s_waitcnt(0xF70);
  lds_barrier();
  for (int c = 0; c < nc; c += 2) {
    SDQ_UP_FILL(As1, Bs1, c + 1);
    SDQ_UP_MUL(As0, Bs0);
    __builtin_amdgcn_s_waitcnt(0xF70);
    lds_barrier();
    if (c + 2 < nc) SDQ_UP_FILL(As0, Bs0, c + 2);
    SDQ_UP_MUL(As1, Bs1);
    __builtin_amdgcn_s_waitcnt(0xF70);
    lds_barrier();
  }
#undef SDQ_UP_FILL
#undef SDQ_UP_MUL
  // Store: sample j -> m = (j / (P-1)) * P + j % (P-1) + 1; rows are contiguous.
  float mx[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) mx[i] = 0.0f;
  const int64_t rbase = r0 + ty * 8;          // 8 rows inside one panel
  const int64_t panel = rbase / kPanel;
  const int lane_row = static_cast<int>(rbase % kPanel);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int jj = j0 + tx * 8 + j;
    if (jj < m_nz) {
      const int m = (jj / (phases - 1)) * phases + jj % (phases - 1) + 1;
      float* dst = xup + (panel * k_up + b * m_up + m) * kPanel + lane_row;
      *reinterpret_cast<float4*>(dst) = make_float4(acc[0][j], acc[1][j], acc[2][j], acc[3][j]);
      *reinterpret_cast<float4*>(dst + 4) = make_float4(acc[4][j], acc[5][j], acc[6][j], acc[7][j]);
#pragma unroll
      for (int i = 0; i < 8; ++i) mx[i] = fmaxf(mx[i], fabsf(acc[i][j]));
    }
  }
  // Reduce the maxima over the 8 threads (tx) that share these rows.
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float val = mx[i];
    val = fmaxf(val, __shfl_xor(val, 1));
    val = fmaxf(val, __shfl_xor(val, 2));
    val = fmaxf(val, __shfl_xor(val, 4));
    mx[i] = val;
  }
  if (tx == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (rbase + i < n) atomicMax(&rmax[rbase + i], __float_as_uint(mx[i]));
  }
}

// One wave per (panel, block) chain set: lane = row.  Words of 32 / bits codes
// never straddle blocks because M is a multiple of 32.  The samples hold
// blocks b0 .. b0 + nb - 1 of the layer (k_up = nb * M per row); codes land at
// their place in the layer's nb_total blocks, the scales are written with
// block 0 and the row's padding words with its last block.
template <int LEVELS>
__global__ __launch_bounds__(64 * kScanWaves) void scan_kernel(
    const float* __restrict__ xup, const uint32_t* __restrict__ rmax, int64_t n, int64_t nb,
    int64_t b0, int64_t nb_total, int64_t k_up, int m_up, int64_t n_chunks,
    uint32_t* __restrict__ codes, float* __restrict__ scales, uint32_t* __restrict__ flag) {
  constexpr int BITS = LEVELS == 2 ? 1 : 2;
  constexpr int PER_WORD = 32 / BITS;
  constexpr int WORDS_PER_CHUNK = 4;
  const int lane = threadIdx.x % 64;
  const int64_t b = static_cast<int64_t>(blockIdx.y) * kScanWaves + threadIdx.x / 64;
  const int64_t panel = blockIdx.x;
  if (b >= nb) return;
  const int64_t gb = b0 + b;            // block index in the layer
  const int64_t r = panel * kPanel + lane;
  const bool live = r < n;
  const float s = live ? __uint_as_float(rmax[r]) : 0.0f;
  if (live && gb == 0) {
    scales[r] = s;
    if (!isfinite(s)) atomicOr(flag, 1u);
  }
  const float theta = s * 0.5f;
  const float* src = xup + (panel * k_up + b * m_up) * kPanel + lane;
  uint32_t* dst_row = codes + (panel * n_chunks * kPanel + lane) * WORDS_PER_CHUNK;
  float u = 0.0f;
  int64_t wj = (gb * m_up) / PER_WORD;  // first word of this block in the row
  for (int m0 = 0; m0 < m_up; m0 += PER_WORD, ++wj) {
    uint32_t word = 0u;
    if (live) {
#pragma unroll 8
      for (int q = 0; q < PER_WORD; ++q) {
        const float x = src[static_cast<int64_t>(m0 + q) * kPanel];
        const float vv = u + x;
        int c;
        if (LEVELS == 3) c = (vv > theta) ? 1 : ((vv < -theta) ? -1 : 0);
        else c = (vv >= 0.0f) ? 1 : -1;
        const float cs = static_cast<float>(c) * s;
        u = vv - cs;
        uint32_t f;
        if (LEVELS == 3) f = c == 0 ? 0u : (c > 0 ? 1u : 3u);
        else f = c > 0 ? 1u : 0u;
        word |= f << (BITS * q);
      }
    }
    const int64_t c = wj / WORDS_PER_CHUNK;
    dst_row[c * kPanel * WORDS_PER_CHUNK + (wj % WORDS_PER_CHUNK)] = word;
  }
  if (gb == nb_total - 1) {
    // Zero the padding words after the last code of the row.
    const int64_t total_words = n_chunks * WORDS_PER_CHUNK;
    for (; wj < total_words; ++wj) {
      const int64_t c = wj / WORDS_PER_CHUNK;
      dst_row[c * kPanel * WORDS_PER_CHUNK + (wj % WORDS_PER_CHUNK)] = 0u;
    }
  }
}

// Base-3 <-> 2-bit fields.  One thread per (row, 80-code chunk): the base-3
// chunk is 16 bytes, the same codes as 2-bit fields are five 32-bit words
// (word i holds codes 16 i .. 16 i + 15, code j of a row at word j / 16 of the
// fields layout).  Code 5p + i of a chunk is field 5p + i of the 160-bit
// string of the five words: bits 10p .. 10p + 9 hold byte p's five fields.
// Consecutive threads take consecutive rows of a panel, so each wave reads
// or writes a chunk of 64 rows as 1 KB contiguous.

// The five fields of a byte of 2-bit fields' string, from the 160-bit string
// held in w[5].
template <int P>
__device__ inline uint32_t ten_bits(const uint32_t (&w)[5]) {
  constexpr int off = 10 * P, wi = off / 32, sh = off % 32;
  uint32_t f = w[wi] >> sh;
  if constexpr (sh > 22) f |= w[wi + 1] << (32 - sh);
  return f & 1023u;
}

template <int P>
__device__ inline void put_ten_bits(uint32_t (&w)[5], uint32_t f) {
  constexpr int off = 10 * P, wi = off / 32, sh = off % 32;
  w[wi] |= f << sh;
  if constexpr (sh > 22) w[wi + 1] |= f >> (32 - sh);
}

// Byte of one group of five fields: digits d = code + 1 (field 00 -> 1,
// 01 -> 2, 11 -> 0), the first code most significant, v = sum d_i 3^(4-i),
// stored as ceil(256 v / 243).
__device__ inline uint32_t base3_byte(uint32_t f) {
  uint32_t v = 0;
#pragma unroll
  for (int i = 0; i < 5; ++i) v = 3u * v + (((f >> (2 * i)) + 1u) & 3u);
  return (256u * v + 242u) / 243u;
}

template <int P>
__device__ inline void repack_byte(const uint32_t (&w)[5], uint32_t (&out)[4]) {
  out[P / 4] |= base3_byte(ten_bits<P>(w)) << (8 * (P % 4));
}

template <int... Ps>
__device__ inline void repack_all(const uint32_t (&w)[5], uint32_t (&out)[4], std::integer_sequence<int, Ps...>) {
  (repack_byte<Ps>(w, out), ...);
}

// Four base-3 slots per thread (the inverse of the unpack below): five whole
// 2-bit chunks (20 field words, 320 codes) in, four 16-byte slots out, each
// access 1 KB contiguous per wave.  total = n_pad * ceil(nch3 / 4); field
// words past the last chunk are padding (code 0); rows past n get zero bytes.
__global__ void repack_base3_kernel(const uint4* __restrict__ fields, int64_t n, int64_t nch2,
                                    int64_t nch3, int64_t quads, int64_t total, uint4* __restrict__ out) {
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t rr = e % kPanel;
    const int64_t g4 = (e / kPanel) % quads;
    const int64_t pn = e / (kPanel * quads);
    const bool row_ok = pn * kPanel + rr < n;
    uint32_t f[20];
#pragma unroll
    for (int c = 0; c < 5; ++c) {
      const int64_t chunk = 5 * g4 + c;
      const uint4 v = row_ok && chunk < nch2 ? fields[(pn * nch2 + chunk) * kPanel + rr]
                                             : make_uint4(0u, 0u, 0u, 0u);
      f[4 * c] = v.x; f[4 * c + 1] = v.y; f[4 * c + 2] = v.z; f[4 * c + 3] = v.w;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t g = 4 * g4 + j;
      if (g >= nch3) break;
      uint32_t o[4] = {0u, 0u, 0u, 0u};
      if (row_ok) {
        const uint32_t w[5] = {f[5 * j], f[5 * j + 1], f[5 * j + 2], f[5 * j + 3], f[5 * j + 4]};
        repack_all(w, o, std::make_integer_sequence<int, 16>{});
      }
      out[(pn * nch3 + g) * kPanel + rr] = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

template <int P>
__device__ inline void unpack_byte(const uint32_t (&by)[4], const uint32_t* pat, uint32_t (&w)[5]) {
  put_ten_bits<P>(w, pat[(by[P / 4] >> (8 * (P % 4))) & 255u]);
}

template <int... Ps>
__device__ inline void unpack_all(const uint32_t (&by)[4], const uint32_t* pat, uint32_t (&w)[5],
                                  std::integer_sequence<int, Ps...>) {
  (unpack_byte<Ps>(by, pat, w), ...);
}

// Four base-3 groups (16 bytes, 80 codes each) per thread: 320 codes are
// exactly five 2-bit chunks of four words, so every load and every store is
// one whole 16-byte slot (a wave's accesses are 1 KB contiguous).  quads =
// ceil(groups / 4) with groups = max(nch3, ceil(4 nch2 / 5)), so every chunk
// of the field layout is written; groups past nch3 and rows past n give
// zero fields.
__global__ __launch_bounds__(256) void unpack_base3_kernel(const uint4* __restrict__ b3, int64_t n,
                                                           int64_t nch2, int64_t nch3, int64_t quads,
                                                           int64_t total, uint4* __restrict__ fields) {
  // Byte -> its five codes as 2-bit fields: digit i of q is the integer part
  // of 3 r after i + 1 steps of r <- fraction part of 3 r, from r = q / 256.
  __shared__ uint32_t pat[256];
  {
    uint32_t r = threadIdx.x, f = 0;
#pragma unroll
    for (int i = 0; i < 5; ++i) {
      r *= 3u;
      f |= (((r >> 8) + 3u) & 3u) << (2 * i);        // digit 0, 1, 2 -> field 11, 00, 01
      r &= 255u;
    }
    pat[threadIdx.x] = f;
  }
  __syncthreads();
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < total;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t rr = e % kPanel;
    const int64_t g4 = (e / kPanel) % quads;
    const int64_t pn = e / (kPanel * quads);
    const bool row_ok = pn * kPanel + rr < n;
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t g = 4 * g4 + j;
      v[j] = row_ok && g < nch3 ? b3[(pn * nch3 + g) * kPanel + rr] : make_uint4(0u, 0u, 0u, 0u);
    }
    uint32_t w[4][5];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int i = 0; i < 5; ++i) w[j][i] = 0u;
      // Slots past nch3 and rows past n are not read: their fields stay zero
      // (code 0), where unpacking a zero byte would give five -1 codes.
      const int64_t g = 4 * g4 + j;
      if (row_ok && g < nch3) {
        const uint32_t by[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
        unpack_all(by, pat, w[j], std::make_integer_sequence<int, 16>{});
      }
    }
#pragma unroll
    for (int c = 0; c < 5; ++c) {
      const int64_t chunk = 5 * g4 + c;
      if (chunk < nch2) {
        uint32_t o[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) o[t] = w[(4 * c + t) / 5][(4 * c + t) % 5];
        fields[(pn * nch2 + chunk) * kPanel + rr] = make_uint4(o[0], o[1], o[2], o[3]);
      }
    }
  }
}

}  // namespace

sdq_status launch_unpack_base3(const void* codes, const sdq_layout* L, uint32_t* fields, hipStream_t stream) {
  const sdq_layout F = fields_view(L);
  const int64_t groups = std::max<int64_t>(L->n_chunks, (4 * F.n_chunks + 4) / 5);
  const int64_t quads = (groups + 3) / 4;
  const int64_t total = L->n_pad * quads;
  const unsigned grid = static_cast<unsigned>(std::min<int64_t>((total + 255) / 256, 16384));
  unpack_base3_kernel<<<grid, 256, 0, stream>>>(static_cast<const uint4*>(codes), L->n, F.n_chunks, L->n_chunks,
                                                quads, total, reinterpret_cast<uint4*>(fields));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "base-3 unpack launch");
  return SDQ_OK;
}

sdq_status launch_encode_blocks(const float* w, int64_t ldw, int64_t b0, int64_t nbl,
                                const sdq_layout* L, const Tables* T, void* codes, float* scales,
                                const QuantWs& ws, uint32_t* rmax_acc, const uint32_t* rmax_scale,
                                hipStream_t stream) {
  const int64_t n_panels = L->n_pad / kPanel;
  const int64_t n_ws = quant_ws_rows(L);     // rows covered by the upsample tiles
  const int B = L->block;
  const int64_t k_up = nbl * L->m_up;        // samples per row held in the workspace
  const float inv_sqrt_b =
      L->hadamard == SDQ_HAD_NONE ? 1.0f : static_cast<float>(1.0 / std::sqrt(static_cast<double>(B)));
  SignMask sm;
  for (int i = 0; i < 8; ++i) sm.w[i] = L->hadamard == SDQ_HAD_SIGNED ? L->had_signs[i] : 0u;
  const dim3 rgrid(static_cast<unsigned>(n_ws / kPanel), static_cast<unsigned>(nbl));
#define SDQ_ROT(BB)                                                                                 \
  rotate_kernel<BB><<<rgrid, dim3(kRotThreads), 0, stream>>>(                                       \
      w, L->n, ldw, n_ws, k_up, L->m_up, T->g0, T->phases, L->hadamard, sm, inv_sqrt_b, ws.v, ws.xup, \
      rmax_acc, ws.flag)
  switch (B) {
    case 64: SDQ_ROT(64); break;
    case 128: SDQ_ROT(128); break;
    default: SDQ_ROT(256); break;
  }
#undef SDQ_ROT
  if (T->m_nz > 0) {
    const dim3 ugrid(static_cast<unsigned>(n_ws / kUpBM),
                     static_cast<unsigned>(T->m_nz_pad / kUpBN), static_cast<unsigned>(nbl));
    upsample_kernel<<<ugrid, dim3(kUpThreads), 0, stream>>>(
        ws.v, T->unz, L->n, n_ws, k_up, B, L->m_up, T->phases, T->m_nz, T->m_nz_pad, ws.xup,
        rmax_acc);
  }
  const dim3 sgrid(static_cast<unsigned>(n_panels), static_cast<unsigned>((nbl + kScanWaves - 1) / kScanWaves));
  if (L->levels == 3)
    scan_kernel<3><<<sgrid, dim3(64 * kScanWaves), 0, stream>>>(
        ws.xup, rmax_scale, L->n, nbl, b0, L->nb, k_up, L->m_up, L->n_chunks,
        static_cast<uint32_t*>(codes), scales, ws.flag);
  else
    scan_kernel<2><<<sgrid, dim3(64 * kScanWaves), 0, stream>>>(
        ws.xup, rmax_scale, L->n, nbl, b0, L->nb, k_up, L->m_up, L->n_chunks,
        static_cast<uint32_t*>(codes), scales, ws.flag);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "encoder launch");
  return SDQ_OK;
}

void clear_rmax(const QuantWs& ws, const sdq_layout* L, hipStream_t stream) {
  clear_kernel<<<dim3(static_cast<unsigned>((L->n_pad + 255) / 256)), dim3(256), 0, stream>>>(
      ws.flag, ws.rmax, L->n_pad);
}

sdq_status launch_quantize(const float* w, const sdq_layout* L, const Tables* T, void* codes,
                           float* scales, const QuantWs& ws, hipStream_t stream) {
  clear_rmax(ws, L, stream);
  if (L->packing != SDQ_PACK_BASE3)
    return launch_encode_blocks(w, L->k, 0, L->nb, L, T, codes, scales, ws, ws.rmax, ws.rmax, stream);
  // Base-3: scan into 2-bit fields in the workspace, then repack.
  const sdq_layout F = fields_view(L);
  sdq_status st = launch_encode_blocks(w, L->k, 0, L->nb, &F, T, ws.codes2, scales, ws, ws.rmax, ws.rmax, stream);
  if (st != SDQ_OK) return st;
  return launch_repack_base3(ws.codes2, L, codes, stream);
}

sdq_status launch_repack_base3(const uint32_t* fields, const sdq_layout* L, void* codes, hipStream_t stream) {
  const sdq_layout F = fields_view(L);
  const int64_t quads = (L->n_chunks + 3) / 4;
  const int64_t total = L->n_pad * quads;
  const unsigned grid = static_cast<unsigned>(std::min<int64_t>((total + 255) / 256, 16384));
  repack_base3_kernel<<<grid, 256, 0, stream>>>(reinterpret_cast<const uint4*>(fields), L->n, F.n_chunks,
                                                L->n_chunks, quads, total, static_cast<uint4*>(codes));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "base-3 repack launch");
  return SDQ_OK;
}

}  // namespace sdq
