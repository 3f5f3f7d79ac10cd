// Internal declarations shared by the libsdq host code and kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/sdq.h"

namespace sdq {

constexpr int kPanel = 64;        // rows per panel of the packed format
constexpr int kChunkBytes = 16;   // bytes per chunk of the packed format
constexpr int kBase3PerChunk = 80; // ternary codes per chunk with base-3 packing

// The same layout with 2-bit ternary fields (base-3 layouts are unpacked to
// it for the paths that read 2-bit fields).
inline sdq_layout fields_view(const sdq_layout* L) {
  sdq_layout F = *L;
  if (F.packing == SDQ_PACK_BASE3) {
    F.packing = SDQ_PACK_FIELDS;
    F.codes_per_chunk = kChunkBytes * 8 / F.bits;
    F.n_chunks = (F.k_up + F.codes_per_chunk - 1) / F.codes_per_chunk;
  }
  return F;
}
inline size_t fields_codes_bytes(const sdq_layout* L) {
  const sdq_layout F = fields_view(L);
  return static_cast<size_t>(F.n_pad) * F.n_chunks * kChunkBytes;
}

// Device coefficient tables for one (block, M, Had) choice on one device.
struct Tables {
  int block = 0;
  int m_up = 0;
  int hadamard = SDQ_HAD_SYLVESTER;   // Had (sdq_hadamard) folded into E
  uint32_t signs[8] = {};              // SDQ_HAD_SIGNED: bit t set <=> s_t = -1
  int g0 = 0;          // gcd(B, M): number of samples whose kernel is a unit impulse
  int phases = 0;      // P = M / g0: samples m with m % P == 0 copy v[(m / P) * (B / g0)]
  int m_nz = 0;        // M - g0 samples per block computed as dense sums
  int m_nz_pad = 0;    // m_nz rounded up to the upsample tile width
  float* unz = nullptr;   // [B][m_nz_pad] fp32 coefficients g(p(t, m_j)), zero padded
  // E = Had D^T (B x M) with D the decimation (Resample back to B), so that
  // x_tilde_b = x_b E (Had = H_B / sqrt(B), diag(s) H_B / sqrt(B) or I).  Two copies:
  //   edec   fp32, groups of four t: edec[((t / 4) * m_pad + m) * 4 + t % 4] =
  //          E[t][m], columns m_up .. m_pad-1 zero (m_pad = M rounded up to 64);
  //   et_hi, et_lo  transposed [M][B] as an fp16 pair hi + lo with
  //          hi = fp16(E) and lo = fp16(E - hi).
  int m_pad = 0;
  float e1max = 0.0f;  // >= max over m of sum_t |E[t][m]| (fp32 table values)
  float* edec = nullptr;
  uint16_t* et_hi = nullptr;
  uint16_t* et_lo = nullptr;
  double* e64 = nullptr;   // E[t][m], fp64, row-major B x M (block reconstruction)
};

// Returns the cached tables of the layout's (block, M, Had) for the current
// device (creating them on first use).
sdq_status get_tables(const sdq_layout* L, const Tables** out);
// The same lookup without creating anything: SDQ_ERR_UNSUPPORTED when the
// tables have not been built on the current device.
sdq_status find_tables(const sdq_layout* L, const Tables** out);

// The body of sdq_linear on a given workspace; may_allocate = false looks the
// coefficient tables up without building them.  linear_ws_need: the bytes
// that workspace needs (0 for an invalid layout or m <= 0).
sdq_status linear_impl(const void* x, sdq_dtype xt, int64_t m, const void* codes, const float* scales,
                       const sdq_layout* L, float* y, int32_t accumulate, void* ws, size_t ws_bytes,
                       void* stream, bool may_allocate);
size_t linear_ws_need(const sdq_layout* L, int64_t m);

// Host fp64 coefficient helpers (also back the parity entry points).
double upsample_kernel(int64_t p, int block, int m_up);          // g(p)
double downsample_entry(int64_t m, int64_t t, int block, int m_up);  // D[m][t]

sdq_status set_error(sdq_status st, const char* fmt, ...);
sdq_status hip_error(hipError_t e, const char* what);

// Workspace carving for sdq_quantize.
// n_ws = n rounded up to 128 rows: the row extent of the rotated and
// upsampled buffers (the upsample kernel works on 128-row tiles).
struct QuantWs {
  uint32_t* flag;    // [0]: non-finite flag
  uint32_t* rmax;    // [n_pad] row maxima as fp32 bit patterns
  float* v;          // [nb][B][n_ws] rotated weights, rows contiguous
  float* xup;        // [n_ws / 64][k_up][64] upsampled samples
  uint32_t* codes2;  // base-3 layouts: the codes as 2-bit fields before repacking (else null)
};
inline int64_t quant_ws_rows(const sdq_layout* L) { return (L->n + 127) / 128 * 128; }
size_t quant_ws_layout(const sdq_layout* L, QuantWs* ws, void* base);

// Zeroes the non-finite flag and the row maxima of ws.
void clear_rmax(const QuantWs& ws, const sdq_layout* L, hipStream_t stream);
sdq_status launch_quantize(const float* w, const sdq_layout* L, const Tables* T, void* codes,
                           float* scales, const QuantWs& ws, hipStream_t stream);
// Base-3 bytes of a ternary layout L from its codes as 2-bit fields (the
// layout fields_view(L)).
sdq_status launch_repack_base3(const uint32_t* fields, const sdq_layout* L, void* codes, hipStream_t stream);
// The inverse: 2-bit fields (fields_view(L)) from base-3 codes.
sdq_status launch_unpack_base3(const void* codes, const sdq_layout* L, uint32_t* fields, hipStream_t stream);
// Encode blocks b0 .. b0 + nbl - 1 from w (row stride ldw; column 0 of w is the
// first column of block b0): rotate and upsample fold their row maxima into
// rmax_acc, the scan uses the row scales in rmax_scale (one buffer for a plain
// encode; a scratch buffer and the fixed scales for a re-encoded block).
sdq_status launch_encode_blocks(const float* w, int64_t ldw, int64_t b0, int64_t nbl,
                                const sdq_layout* L, const Tables* T, void* codes, float* scales,
                                const QuantWs& ws, uint32_t* rmax_acc, const uint32_t* rmax_scale,
                                hipStream_t stream);

// The linears one contraction launch covers (sdq_linear: one; sdq_linear_group:
// up to kMaxGroup).  They share the input and the layout's k, block, M, levels,
// Had and packing (the expansion), and have their own rows, codes, scales and
// outputs.  Passed to the kernels by value; a workgroup finds its linear from
// its place in the launch (the prefix sums `first` of the units -- panel
// groups, panels or column tiles -- each linear contributes).
constexpr int kMaxGroup = 4;
struct LinearSet {
  int count = 0;
  const void* codes[kMaxGroup] = {};
  const float* scales[kMaxGroup] = {};
  float* y[kMaxGroup] = {};
  int64_t n[kMaxGroup] = {};
  int64_t first[kMaxGroup + 1] = {};   // filled by the launcher for its unit
};
// Rows over all linears of the set, rounded up to whole panels per linear.
inline int64_t set_panels(const LinearSet& S) {
  int64_t p = 0;
  for (int j = 0; j < S.count; ++j) p += (S.n[j] + kPanel - 1) / kPanel;
  return p;
}

// Compute units of the current device (cached per device; 256 if unknown).
int64_t device_compute_units();

// Decode path (m <= 16): expansion (fp32 x_tilde) then LUT GEMV.
size_t decode_ws_bytes(const sdq_layout* L, int64_t m);
sdq_status decode_supported(const sdq_layout* L);
// When the GEMV splits K it accumulates into y atomically; y must then start
// at zero (or hold the values to accumulate onto): the expansion zeroes it if
// handed the set (zero), else the GEMV launch does unless y_ready is set.
// `panels`: the panels of the whole set (the split depends on the grid size).
bool decode_needs_zero_y(const sdq_layout* L, int64_t m, int64_t panels);
// Whether the decode path reads base-3 codes as stored (one activation row,
// table GEMV); every other path reads them unpacked to fields_view(L).
bool decode_reads_base3(const sdq_layout* L, int64_t m);
sdq_status launch_decode_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                const Tables* T, void* ws, const LinearSet* zero, hipStream_t stream);
// accumulate: y += result instead of y = result.
sdq_status launch_decode_contract(int64_t m, LinearSet set, const sdq_layout* L, bool accumulate, void* ws,
                                  bool y_ready, hipStream_t stream);

// Prefill path (m > 16): expansion (fp16 x_tilde) then MFMA GEMM.  Layouts
// without Had keep x_tilde as an fp16 pair (prefill_split).  The workspace:
// the fp16 x_tilde plane(s) (prefill_planes_bytes), then the per-row powers of
// two p_i [m] and 1 / p_i [m] (fp32) that keep x_tilde inside fp16's range.
bool prefill_split(const sdq_layout* L);
size_t prefill_planes_bytes(const sdq_layout* L, int64_t m);
size_t prefill_ws_bytes(const sdq_layout* L, int64_t m);
sdq_status launch_prefill_expand(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                 const Tables* T, void* ws, hipStream_t stream);
sdq_status launch_prefill_contract(int64_t m, LinearSet set, const sdq_layout* L, bool accumulate, void* ws,
                                   hipStream_t stream);

// Block compensation (Algorithm 1's block loop), fp64.
sdq_status launch_hessian_accumulate(const float* x, int64_t m, int64_t k, double* h, hipStream_t stream);
size_t hessian_factor_ws_bytes(int64_t k);
sdq_status launch_hessian_factor(const double* h, int64_t k, double lam, double* u, void* ws,
                                 hipStream_t stream);
size_t comp_ws_bytes(const sdq_layout* L);
sdq_status launch_quantize_compensated(const float* w, const sdq_layout* L, const Tables* T,
                                       const double* u, int update, void* codes, float* scales, void* ws,
                                       hipStream_t stream);

// Moments (mean, variance) of a device array.
size_t moments_ws_bytes(int64_t count);
sdq_status launch_moments(const float* w, int64_t count, double* out, void* ws, size_t ws_bytes,
                          hipStream_t stream);

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace sdq
