// Prefill path of sdq_linear (m > 16 activation rows), the contraction:
//
//   gemm     y[i, r] = s_r * sum_j x_tilde[i, j] C[r, j]: the codes are expanded
//            in registers to fp16 +1 / 0 / -1 and fed to the fp16 matrix cores
//            (v_mfma_f32_32x32x16_f16, fp32 accumulation).  This is the
//            contraction of Fig. 5 at prefill batch sizes, where it is a dense
//            GEMM over the oversampled length.  x_tilde comes from the
//            expansion in expand_prefill.hip.
//
// MFMA operand convention used here: lane l supplies row (A) or column (B)
// l % 32 and the eight consecutive k of group l / 32.  Any fixed pairing of
// A's and B's k slots gives the same sum, so only the row/column mapping and
// the accumulator layout (row 8*(v/4) + 4*(l/32) + v%4, column l%32 for
// accumulator v) matter.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>
#include <cstdlib>
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


// ---------------------------------------------------------------------------
// GEMM.  Workgroup tile 256 (activation rows) x 256 (weight rows), k step 64.
// Eight waves, 2 (activation rows) x 4 (weight rows), each owning a 128 x 64
// tile (4 x 2 accumulator tiles of 32 x 32), two waves per SIMD; or four
// waves side by side along the weight rows, each owning 256 x 64.  The
// x_tilde tile is double-buffered in LDS and filled straight from global
// memory (global_load_lds_dwordx4, no
// staging registers); its 16-byte groups are XOR-swizzled by row so that the
// fragment reads of 16 consecutive rows fall on distinct banks.  A ring of
// four buffers (128 KB): the copies for step k + 2 are issued while step k
// computes, so a copy has two steps to land.  The codes go from global memory
// to registers two steps ahead as well and are expanded to fp16 with
// byte-permute lookups, each expanded fragment feeding eight MFMAs.
// ---------------------------------------------------------------------------
constexpr int kBM = 256, kBN = 256, kBK = 64;
constexpr int kTileHalves = kBM * kBK;      // one x_tilde tile (32 KB)
constexpr int kABufs = 4;                    // a ring of tiles; steps k + 1 and k + 2 in flight during k

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) const void* gbl_void_ptr;

// 16-byte group g of row r is stored in slot g ^ swz(r).
__device__ inline int swz(int r) { return (r >> 1) & 7; }

// Two ternary codes (4 bits: f0 at bits 0-1, f1 at bits 2-3) -> fp16 pair.
// v_perm_b32 picks each result byte from the table by its selector byte: the
// low bytes of both halves use selector 0x0C (constant 0x00), the high bytes
// use the code field, and table bytes 0..3 of 0xBC003C00 are the fp16 high
// bytes for fields 00, 01, 10, 11.
__device__ inline uint32_t tern_pair(uint32_t nib) {
  const uint32_t sel = 0x000C000Cu | ((nib & 3u) << 8) | ((nib & 0xCu) << 22);
  return __builtin_amdgcn_perm(0u, 0xBC003C00u, sel);
}

// Two binary codes (bits 0, 1; 1 = +1) -> fp16 pair; table bytes 0xBC, 0x3C.
__device__ inline uint32_t bin_pair(uint32_t two) {
  const uint32_t sel = 0x000C000Cu | ((two & 1u) << 8) | ((two & 2u) << 23);
  return __builtin_amdgcn_perm(0u, 0x00003CBCu, sel);
}

template <int LEVELS>
__device__ inline half8 expand8(uint32_t bits) {
  uint32_t d[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) d[q] = LEVELS == 3 ? tern_pair(bits >> (4 * q)) : bin_pair(bits >> (2 * q));
  half8 out;
  __builtin_memcpy(&out, d, 16);
  return out;
}

// The 8 codes this lane feeds at k step ks (0..3) of the current 64-code
// slice, from the slice's words as loaded by load_codes.
template <int LEVELS>
__device__ inline uint32_t codes_at(const uint4& c, int ks, int half) {
  if (LEVELS == 3) {
    const uint32_t w = ks == 0 ? c.x : ks == 1 ? c.y : ks == 2 ? c.z : c.w;
    return (w >> (16 * half)) & 0xFFFFu;
  }
  const uint32_t w = ks < 2 ? c.x : c.y;
  return (w >> (16 * (ks & 1) + 8 * half)) & 0xFFu;
}

// Words holding codes [64*it, 64*it + 64) of weight row col.  Columns past
// the padded row count read the last row: they only feed outputs that are
// never stored.
template <int LEVELS>
__device__ inline uint4 load_codes(const uint4* __restrict__ codes, int64_t col, int64_t n_pad,
                                   int64_t n_chunks, int it) {
  col = col < n_pad ? col : n_pad - 1;
  const int64_t c = LEVELS == 3 ? it : it / 2;
  const uint4 q = codes[((col / kPanel) * n_chunks + c) * kPanel + col % kPanel];
  if (LEVELS == 3) return q;
  return (it & 1) ? make_uint4(q.z, q.w, 0u, 0u) : make_uint4(q.x, q.y, 0u, 0u);
}

// Workgroups are dealt to the eight XCDs round-robin by index, and each XCD
// has its own L2.  Workgroup `id` of `total` takes tile xcd_range(id) of an
// order in which every XCD owns one contiguous range; the order walks pairs of
// row tiles across the column tiles (row tile 2p, 2p + 1 of column tile c are
// neighbours), so the workgroups resident on one XCD at a time cover a block
// of two row tiles by many column tiles and its L2 fetches each x_tilde and
// code slice once for all of them.
constexpr int kXcds = 8;
__device__ inline int64_t xcd_index(int64_t id, int64_t total) {
  const int64_t xcd = id % kXcds, j = id / kXcds;
  const int64_t per = total / kXcds, rem = total % kXcds;
  return xcd * per + (xcd < rem ? xcd : rem) + j;
}
__device__ inline void prefill_tile(int64_t t, int64_t m_tiles, int64_t n_tiles, int64_t* mt, int64_t* nt) {
  const int64_t pair_tiles = 2 * n_tiles;          // tiles of one pair of row tiles
  const int64_t p = t / pair_tiles, r = t % pair_tiles;
  const int64_t rows_in_pair = min<int64_t>(2, m_tiles - 2 * p);
  *nt = r / rows_in_pair;
  *mt = 2 * p + r % rows_in_pair;
}

// row_inv: 1 / p_i of every activation row, the powers of two the expansion
// scaled the rows by; the epilogue multiplies them back out (exact).
// A launch covers the tiles t_base .. t_base + t_count - 1 of that order: NC =
// 2 a whole 256 x 256 tile per workgroup, NC = 1 half of one (256 activation
// rows x 128 weight rows, each wave 32 of them), so that a last, partly
// filled wave of whole tiles can run as one full wave of half tiles.
// W waves: 4 (each 256 activation rows x 64 weight rows, 256 accumulator
// registers, one wave per SIMD) or 8 (each 128 x 64, two waves per SIMD).
template <int LEVELS, int NC, int W>
__global__ __launch_bounds__(64 * W, 1) void gemm_prefill_kernel(
    const _Float16* __restrict__ xt, const float* __restrict__ row_inv, LinearSet S, int64_t m,
    int64_t n_chunks, int64_t k_up_pad, int64_t m_tiles, int64_t n_tiles, int64_t t_base, int64_t t_count,
    int accumulate) {
  __shared__ __attribute__((aligned(1024))) _Float16 As[kABufs][kTileHalves];
  constexpr int RPW = kBM / (W / 4);          // activation rows per wave
  constexpr int RT = RPW / 32;                 // 32-row MFMA tiles per wave
  constexpr int FC = kBM / W / 8;              // tile-fill copies per wave and step (8 rows each)
  const int tid = threadIdx.x;
  const int lane = tid % 64;
  const int wave = tid / 64;
  const int wq = wave % 4;                     // column quarter
  const int row0 = (wave / 4) * RPW;           // first activation row of the wave in the tile
  const int half = lane / 32;
  int64_t mt, nt;
  const int64_t u = xcd_index(blockIdx.x, static_cast<int64_t>(gridDim.x));
  const int nh = NC == 2 ? 0 : static_cast<int>(u % 2);   // which half of the tile's weight rows
  prefill_tile(t_base + (NC == 2 ? u : u / 2), m_tiles, n_tiles, &mt, &nt);
  const int lin = [&] {                           // units: column tiles of kBN weight rows
    int j = 0;
#pragma unroll
    for (int i = 1; i < kMaxGroup; ++i)
      if (i < S.count && nt >= S.first[i]) j = i;
    return j;
  }();
  const int64_t n = S.n[lin];
  const int64_t n_pad = (n + kPanel - 1) / kPanel * kPanel;
  const uint4* __restrict__ codes = static_cast<const uint4*>(S.codes[lin]);
  const float* __restrict__ scales = S.scales[lin];
  float* __restrict__ y = S.y[lin];
  const int64_t m0 = mt * kBM;
  const int64_t n0 = (nt - S.first[lin]) * kBN + (NC == 2 ? wq * 64 : nh * 128 + wq * 32);
  int64_t cols[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) cols[c] = n0 + 32 * c + lane % 32;
  const int n_iter = static_cast<int>(k_up_pad / kBK);

  floatx16 acc[RT][NC];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[r][c][v] = 0.0f;

  // Tile fill: wave w fills rows 64 w .. 64 w + 63 with 8 copies of 1 KB (8
  // rows each); lane l of copy j writes slot l % 8 of row 64 w + 8 j + l / 8,
  // which holds 16-byte group (l % 8) ^ swz(row).  Rows past m read row m - 1:
  // they only feed output rows that are not stored.
  uint32_t a_off[FC];                       // element offsets (m * k_up_pad < 2^31)
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const int r = wave * (kBM / W) + 8 * j + lane / 8;
    const int64_t row = m0 + r;
    a_off[j] = static_cast<uint32_t>((row < m ? row : m - 1) * k_up_pad + 8 * ((lane % 8) ^ swz(r)));
  }
#define SDQ_FILL_A(BUF, IT)                                                                      \
  do {                                                                                           \
    const _Float16* src_ = xt + static_cast<uint32_t>((IT) * kBK);                               \
    _Float16* dst_ = &As[(BUF)][wave * (kBM / W) * kBK];                                         \
    _Pragma("unroll") for (int j = 0; j < FC; ++j)                                               \
      __builtin_amdgcn_global_load_lds((gbl_void_ptr)(src_ + a_off[j]),                          \
                                       (lds_void_ptr)(dst_ + j * 8 * kBK), 16, 0, 0);            \
  } while (0)

  const int it1 = n_iter > 1 ? 1 : 0;
  SDQ_FILL_A(0, 0);
  SDQ_FILL_A(1, it1);
  uint4 c0 = load_codes<LEVELS>(codes, cols[0], n_pad, n_chunks, 0);
  uint4 c1 = load_codes<LEVELS>(codes, cols[NC - 1], n_pad, n_chunks, 0);
  uint4 d0 = load_codes<LEVELS>(codes, cols[0], n_pad, n_chunks, it1);   // the next step's
  uint4 d1 = load_codes<LEVELS>(codes, cols[NC - 1], n_pad, n_chunks, it1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // Fragment read offsets (halves) of row tile rt, k group g: row r = 32 rt + lane % 32.
  const int fr = lane % 32;
  for (int it = 0; it < n_iter; ++it) {
    // Step it reads buffer it % 4 and copies step it + 2 into buffer
    // (it + 2) % 4 = cur ^ 2, an index the compiler can tell apart from cur,
    // so it does not wait for the copies before reading (near the end the
    // last step is copied again; that copy is never read).
    const int cur = it & 3;
    const int n2 = it + 2 < n_iter ? it + 2 : n_iter - 1;
    SDQ_FILL_A(cur ^ 2, n2);
    const uint4 e0 = load_codes<LEVELS>(codes, cols[0], n_pad, n_chunks, n2);
    const uint4 e1 = NC == 2 ? load_codes<LEVELS>(codes, cols[NC - 1], n_pad, n_chunks, n2) : e0;
    const _Float16* abuf = As[cur];
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      half8 b[NC];
      b[0] = expand8<LEVELS>(codes_at<LEVELS>(c0, ks, half));
      if (NC == 2) b[NC - 1] = expand8<LEVELS>(codes_at<LEVELS>(c1, ks, half));
      const int g = 2 * ks + half;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int r = row0 + rt * 32 + fr;
        const half8 afrag = *reinterpret_cast<const half8*>(abuf + r * kBK + 8 * (g ^ swz(r)));
#pragma unroll
        for (int c = 0; c < NC; ++c) acc[rt][c] = mfma32(afrag, b[c], acc[rt][c]);
      }
    }
    c0 = d0;
    c1 = d1;
    d0 = e0;
    d1 = e1;
    // The next step's tile (copied a step ago) has landed for this lane: at
    // most this step's eight tile copies and two code loads are outstanding
    // (vmcnt 10; expcnt and lgkmcnt not waited on), and for every lane after the
    // barrier.  A plain s_barrier: __syncthreads() adds a release fence, which
    // waits for every outstanding LDS copy.  The empty asm statements keep LDS
    // accesses from moving across it; every fragment read of the buffer that
    // is refilled next has returned before its MFMAs issued.
    __builtin_amdgcn_s_waitcnt(W == 4 ? 0xF7A : 0xF70 | (FC + 2));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  }
#undef SDQ_FILL_A

  // The row factors of the tile, staged in the first buffer of the ring once
  // every copy has landed and every fragment read is done (a separate LDS
  // array would make the compiler wait for all copies in every step).
  static_assert(kBM == 256, "one row factor per thread");
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  float* rinv = reinterpret_cast<float*>(&As[0][0]);
  if (tid < kBM) rinv[tid] = m0 + tid < m ? row_inv[m0 + tid] : 1.0f;
  __syncthreads();
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int64_t col = cols[c];
    if (col >= n) continue;
    const float s = scales[col];
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int lr = row0 + r * 32 + 8 * (v / 4) + 4 * half + (v % 4);
        const int64_t row = m0 + lr;
        if (row < m) {
          const float val = acc[r][c][v] * s * rinv[lr];
          y[row * n + col] = accumulate ? y[row * n + col] + val : val;
        }
      }
  }
}


}  // namespace

size_t prefill_planes_bytes(const sdq_layout* L, int64_t m) {
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  return align_up(static_cast<size_t>(m) * k_up_pad * 2, 256) * (prefill_split(L) ? 2 : 1);
}

size_t prefill_ws_bytes(const sdq_layout* L, int64_t m) {
  return prefill_planes_bytes(L, m) + align_up(static_cast<size_t>(m) * 2 * sizeof(float), 256);
}

sdq_status launch_prefill_contract(int64_t m, LinearSet S, const sdq_layout* L, bool accumulate, void* ws,
                                   hipStream_t stream) {
  S.first[0] = 0;
  for (int j = 0; j < S.count; ++j) S.first[j + 1] = S.first[j] + (S.n[j] + kBN - 1) / kBN;
  for (int j = S.count + 1; j <= kMaxGroup; ++j) S.first[j] = S.first[S.count];
  const int64_t n_tiles = S.first[S.count];
  const int64_t k_up_pad = L->n_chunks * L->codes_per_chunk;
  const size_t plane = align_up(static_cast<size_t>(m) * k_up_pad * 2, 256);
  const float* row_inv = reinterpret_cast<const float*>(static_cast<const char*>(ws) + prefill_planes_bytes(L, m)) + m;
  // The kernel addresses x_tilde with 32-bit element offsets: launch row
  // chunks of at most 2^31 elements.
  const int64_t rows_max = std::max<int64_t>(kBM, ((int64_t{1} << 31) / k_up_pad) / kBM * kBM);
  const int passes = prefill_split(L) ? 2 : 1;   // x_tilde hi, then lo added on
  const int64_t cus = device_compute_units();
  // Eight waves (two per SIMD, so one wave's LDS and memory waits overlap the
  // other's MFMAs) by default: measured 431 against 437-445 us on 8192x8192 and
  // 1489 against 1540-1548 us on 28672x8192 at m = 2048, equal on 8192x28672.
  // SDQ_PF_WAVES=4 selects one wave per SIMD (a tuning aid).
  static const char* env_w = std::getenv("SDQ_PF_WAVES");
  const int waves = env_w && std::atoi(env_w) == 4 ? 4 : 8;
  for (int pass = 0; pass < passes; ++pass) {
    const _Float16* xbuf = reinterpret_cast<const _Float16*>(static_cast<const char*>(ws) + pass * plane);
    const int acc = accumulate || pass > 0 ? 1 : 0;
    for (int64_t r0 = 0; r0 < m; r0 += rows_max) {
      const int64_t mm = std::min(rows_max, m - r0);
      const int64_t m_tiles = (mm + kBM - 1) / kBM;
      const _Float16* xc = xbuf + r0 * k_up_pad;
      LinearSet Sc = S;
      for (int j = 0; j < S.count; ++j) Sc.y[j] = S.y[j] + r0 * S.n[j];
      // One workgroup per CU: whole tiles in full waves, and a last wave that
      // would be at most half full as twice as many half tiles (same time per
      // wave of work, no idle half).
      const int64_t tiles = m_tiles * n_tiles;
      const int64_t tail = tiles % cus;
      const int64_t t_half = tail > 0 && 2 * tail <= cus ? tail : 0;
      const int64_t t_whole = tiles - t_half;
      auto launch = [&](auto lv, auto nc, int64_t t_base, int64_t t_count) {
        constexpr int LV = decltype(lv)::value, NC = decltype(nc)::value;
        if (t_count <= 0) return;
        const dim3 ggrid(static_cast<unsigned>(t_count * (NC == 2 ? 1 : 2)));
        if (waves == 8)
          gemm_prefill_kernel<LV, NC, 8><<<ggrid, dim3(512), 0, stream>>>(xc, row_inv + r0, Sc, mm, L->n_chunks,
                                                                        k_up_pad, m_tiles, n_tiles, t_base,
                                                                        t_count, acc);
        else
          gemm_prefill_kernel<LV, NC, 4><<<ggrid, dim3(256), 0, stream>>>(xc, row_inv + r0, Sc, mm, L->n_chunks,
                                                                        k_up_pad, m_tiles, n_tiles, t_base,
                                                                        t_count, acc);
      };
      using L2_ = std::integral_constant<int, 2>;
      using L3_ = std::integral_constant<int, 3>;
      using W_ = std::integral_constant<int, 2>;
      using H_ = std::integral_constant<int, 1>;
      if (L->levels == 2) {
        launch(L2_{}, W_{}, 0, t_whole);
        launch(L2_{}, H_{}, t_whole, t_half);
      } else {
        launch(L3_{}, W_{}, 0, t_whole);
        launch(L3_{}, H_{}, t_whole, t_half);
      }
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "prefill GEMM launch");
  return SDQ_OK;
}

// Compute units of the current device (cached per device).
int64_t device_compute_units() {
  static int64_t cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cached[dev] = v;
  }
  return cached[dev];
}

}  // namespace sdq
