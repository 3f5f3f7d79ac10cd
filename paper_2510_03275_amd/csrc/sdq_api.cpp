// libsdq host side: argument validation, geometry, coefficient tables,
// MultiOSR allocation and dispatch to the HIP kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <array>
#include <map>
#include <mutex>
#include <numeric>
#include <string>
#include <tuple>
#include <vector>

#include "sdq_internal.h"

namespace sdq {

static thread_local std::string g_last_error;

sdq_status set_error(sdq_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

sdq_status hip_error(hipError_t e, const char* what) {
  return set_error(SDQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// Coefficients.  The upsampling Resample of Algorithm 1 is the band-limited
// periodic interpolation of the block; output sample m sits at position
// m*B/M of the input grid, so its weight on input t is the periodic sinc
// evaluated at tau = (m*B - t*M)/M (taken mod B).  Decimation (Resample back
// to B) has the analogous closed form with the folded Nyquist term.
// ---------------------------------------------------------------------------
double upsample_kernel(int64_t p, int block, int m_up) {
  if (p == 0) return 1.0;
  if (p % m_up == 0) return 0.0;
  const double tau = static_cast<double>(p) / static_cast<double>(m_up);
  return std::sin(M_PI * tau) / (static_cast<double>(block) * std::tan(M_PI * tau / block));
}

double downsample_entry(int64_t m, int64_t t, int block, int m_up) {
  if (m_up == block) return m == t ? 1.0 : 0.0;
  const int64_t num = m * block - t * m_up;
  double val;
  if (num % m_up == 0) {
    const int64_t k = num / m_up;
    val = ((k % block == 0) ? static_cast<double>(block) : 0.0) + ((k % 2 == 0) ? 1.0 : -1.0);
  } else {
    const double tau = static_cast<double>(num) / static_cast<double>(m_up);
    val = std::sin(M_PI * tau) / std::tan(M_PI * tau / block) + std::cos(M_PI * tau);
  }
  return val / m_up;
}

static int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    const int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

constexpr int kUpsampleTileN = 64;   // column tile of the upsampling kernel

using SignWords = std::array<uint32_t, 8>;
static std::mutex g_tables_mutex;
static std::map<std::tuple<int, int, int, int, SignWords>, Tables> g_tables;

static sdq_status get_tables_for(int block, int m_up, int had, const SignWords& signs,
                                 const Tables** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_tables_mutex);
  auto key = std::make_tuple(dev, block, m_up, had, signs);
  auto it = g_tables.find(key);
  if (it != g_tables.end()) {
    *out = &it->second;
    return SDQ_OK;
  }
  Tables T;
  T.block = block;
  T.m_up = m_up;
  T.hadamard = had;
  std::copy(signs.begin(), signs.end(), T.signs);
  T.g0 = static_cast<int>(gcd64(block, m_up));
  T.phases = m_up / T.g0;
  T.m_nz = m_up - T.g0;
  T.m_nz_pad = (T.m_nz + kUpsampleTileN - 1) / kUpsampleTileN * kUpsampleTileN;
  // fp32 kernel values indexed by p = (m*B - t*M) mod (B*M): rounded once from fp64.
  const int64_t bm = static_cast<int64_t>(block) * m_up;
  std::vector<float> unz(static_cast<size_t>(block) * std::max(T.m_nz_pad, 1), 0.0f);
  for (int t = 0; t < block; ++t) {
    int j = 0;
    for (int m = 0; m < m_up; ++m) {
      if (m % T.phases == 0) continue;   // unit-impulse samples are copied, not summed
      const int64_t p = ((static_cast<int64_t>(m) * block - static_cast<int64_t>(t) * m_up) % bm + bm) % bm;
      unz[static_cast<size_t>(t) * T.m_nz_pad + j] = static_cast<float>(upsample_kernel(p, block, m_up));
      ++j;
    }
  }
  // E^T[m][t] = sum_u Had[t][u] D[m][u]: a Walsh-Hadamard transform of each row
  // of D (fp64), scaled by 1/sqrt(B), its entry t negated where s_t = -1 for
  // the signed Had, or D itself without Had; kept in fp32 and as two fp16 terms.
  const size_t em = static_cast<size_t>(m_up) * block;
  T.m_pad = (m_up + 63) / 64 * 64;
  std::vector<float> edec(static_cast<size_t>(T.m_pad) * block, 0.0f);
  std::vector<uint16_t> eh(em), el(em);
  std::vector<double> e64(em);          // E[t][m] in fp64, row-major B x M
  std::vector<double> row(block);
  const double inv_sqrt_b = 1.0 / std::sqrt(static_cast<double>(block));
  double e1max = 0.0;   // max over samples m of sum_t |fp32(E[t][m])|
  for (int m = 0; m < m_up; ++m) {
    for (int t = 0; t < block; ++t) row[t] = downsample_entry(m, t, block, m_up);
    if (had != SDQ_HAD_NONE) {
      for (int h = 1; h < block; h <<= 1)
        for (int i = 0; i < block; i += 2 * h)
          for (int j = i; j < i + h; ++j) {
            const double a = row[j], c = row[j + h];
            row[j] = a + c;
            row[j + h] = a - c;
          }
      for (int t = 0; t < block; ++t) {
        row[t] *= inv_sqrt_b;
        if (had == SDQ_HAD_SIGNED && (signs[t / 32] >> (t % 32) & 1u)) row[t] = -row[t];
      }
    }
    double col1 = 0.0;
    for (int t = 0; t < block; ++t) {
      const double val = row[t];
      const size_t at = static_cast<size_t>(m) * block + t;
      e64[static_cast<size_t>(t) * m_up + m] = val;
      edec[(static_cast<size_t>(t / 4) * T.m_pad + m) * 4 + t % 4] = static_cast<float>(val);
      col1 += std::fabs(static_cast<double>(static_cast<float>(val)));
      const _Float16 hi = static_cast<_Float16>(val);
      const _Float16 lo = static_cast<_Float16>(val - static_cast<double>(hi));
      std::memcpy(&eh[at], &hi, 2);
      std::memcpy(&el[at], &lo, 2);
    }
    e1max = std::max(e1max, col1);
  }
  // Rounded up to fp32 (with a relative margin) so that |x_b E[:, m]| <=
  // max|x_b| * e1max holds for the device's fp32 sums.
  T.e1max = std::nextafter(static_cast<float>(e1max * (1.0 + 1e-6)), INFINITY);
  // Device copies; on any failure the tables allocated so far are freed.
  auto fail = [&](sdq_status st, const char* what, hipError_t err) {
    for (void* ptr : {static_cast<void*>(T.unz), static_cast<void*>(T.edec), static_cast<void*>(T.et_hi),
                      static_cast<void*>(T.et_lo), static_cast<void*>(T.e64)})
      if (ptr) (void)hipFree(ptr);
    return st == SDQ_ERR_NOMEM ? set_error(st, "%s: %s", what, hipGetErrorString(err)) : hip_error(err, what);
  };
  if (T.m_nz > 0) {
    e = hipMalloc(&T.unz, unz.size() * sizeof(float));
    if (e != hipSuccess) return fail(SDQ_ERR_NOMEM, "table allocation", e);
  }
  e = hipMalloc(&T.edec, edec.size() * 4);
  if (e == hipSuccess) e = hipMalloc(&T.et_hi, em * 2);
  if (e == hipSuccess) e = hipMalloc(&T.et_lo, em * 2);
  if (e == hipSuccess) e = hipMalloc(&T.e64, em * 8);
  if (e != hipSuccess) return fail(SDQ_ERR_NOMEM, "table allocation", e);
  if (T.m_nz > 0) e = hipMemcpy(T.unz, unz.data(), unz.size() * sizeof(float), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(T.edec, edec.data(), edec.size() * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(T.et_hi, eh.data(), em * 2, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(T.et_lo, el.data(), em * 2, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(T.e64, e64.data(), em * 8, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(SDQ_ERR_HIP, "table upload", e);
  auto res = g_tables.emplace(key, T);
  *out = &res.first->second;
  return SDQ_OK;
}

sdq_status get_tables(const sdq_layout* L, const Tables** out) {
  SignWords w{};
  if (L->hadamard == SDQ_HAD_SIGNED) std::copy(L->had_signs, L->had_signs + 8, w.begin());
  return get_tables_for(L->block, L->m_up, L->hadamard, w, out);
}

sdq_status find_tables(const sdq_layout* L, const Tables** out) {
  SignWords w{};
  if (L->hadamard == SDQ_HAD_SIGNED) std::copy(L->had_signs, L->had_signs + 8, w.begin());
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_tables_mutex);
  auto it = g_tables.find(std::make_tuple(dev, L->block, L->m_up, L->hadamard, w));
  if (it == g_tables.end())
    return set_error(SDQ_ERR_UNSUPPORTED, "the coefficient tables of this layout are not on the current device: "
                                          "call sdq_prepare_layout first");
  *out = &it->second;
  return SDQ_OK;
}

static bool valid_block(int b) { return b == 64 || b == 128 || b == 256; }

// The Had choice: a known mode, sign bits only below the block for the
// signed Had and none otherwise.
static bool valid_hadamard(const sdq_layout* L) {
  if (L->hadamard != SDQ_HAD_NONE && L->hadamard != SDQ_HAD_SYLVESTER && L->hadamard != SDQ_HAD_SIGNED)
    return false;
  for (int i = 0; i < 8; ++i) {
    const uint32_t allowed = L->hadamard != SDQ_HAD_SIGNED || 32 * i >= L->block ? 0u
                             : (32 * (i + 1) <= L->block ? ~0u : (1u << (L->block - 32 * i)) - 1u);
    if (L->had_signs[i] & ~allowed) return false;
  }
  return true;
}

static sdq_status check_layout(const sdq_layout* L) {
  if (!L) return set_error(SDQ_ERR_ARG, "layout is NULL");
  if (L->n < 0 || L->k <= 0 || !valid_block(L->block) || L->k % L->block ||
      (L->levels != 2 && L->levels != 3) || L->m_up < L->block || L->m_up % 32 ||
      L->nb != L->k / L->block || L->k_up != L->nb * L->m_up ||
      L->bits != (L->levels == 2 ? 1 : 2) ||
      (L->packing != SDQ_PACK_FIELDS && L->packing != SDQ_PACK_BASE3) ||
      (L->packing == SDQ_PACK_BASE3 && L->levels != 3) ||
      L->codes_per_chunk != (L->packing == SDQ_PACK_BASE3 ? kBase3PerChunk : kChunkBytes * 8 / L->bits) ||
      L->n_chunks != (L->k_up + L->codes_per_chunk - 1) / L->codes_per_chunk ||
      L->n_pad != (L->n + kPanel - 1) / kPanel * kPanel || !valid_hadamard(L))
    return set_error(SDQ_ERR_ARG, "layout is not one produced by sdq_layout_init");
  return SDQ_OK;
}

size_t quant_ws_layout(const sdq_layout* L, QuantWs* ws, void* base) {
  char* p = static_cast<char*>(base);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return p ? p + at : nullptr;
  };
  QuantWs w;
  w.flag = reinterpret_cast<uint32_t*>(take(256));
  w.rmax = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(L->n_pad) * 4));
  const size_t rows = static_cast<size_t>(quant_ws_rows(L));
  w.v = reinterpret_cast<float*>(take(rows * L->k * 4));
  w.xup = reinterpret_cast<float*>(take(rows * L->k_up * 4));
  w.codes2 = L->packing == SDQ_PACK_BASE3 ? reinterpret_cast<uint32_t*>(take(fields_codes_bytes(L))) : nullptr;
  if (ws) *ws = w;
  return off;
}

}  // namespace sdq

using namespace sdq;

extern "C" {

int32_t sdq_version(void) { return 100; }

const char* sdq_status_string(sdq_status s) {
  switch (s) {
    case SDQ_OK: return "ok";
    case SDQ_ERR_ARG: return "invalid argument";
    case SDQ_ERR_SHAPE: return "unsupported shape";
    case SDQ_ERR_OSR: return "unsupported oversampling ratio";
    case SDQ_ERR_LEVELS: return "levels must be 2 or 3";
    case SDQ_ERR_NONFINITE: return "non-finite weight";
    case SDQ_ERR_WORKSPACE: return "workspace missing or too small";
    case SDQ_ERR_HIP: return "HIP runtime error";
    case SDQ_ERR_NOMEM: return "out of device memory";
    case SDQ_ERR_UNSUPPORTED: return "unsupported request";
    case SDQ_ERR_NOT_SPD: return "matrix not positive definite";
  }
  return "unknown status";
}

const char* sdq_last_error(void) { return g_last_error.c_str(); }

sdq_status sdq_layout_init(sdq_layout* out, int64_t n, int64_t k, double osr, int32_t levels,
                           int32_t block) {
  if (!out) return set_error(SDQ_ERR_ARG, "out is NULL");
  if (block == 0) block = 256;
  if (n < 0 || k <= 0) return set_error(SDQ_ERR_ARG, "need n >= 0 and k > 0 (n=%lld k=%lld)",
                                        (long long)n, (long long)k);
  if (!valid_block(block)) return set_error(SDQ_ERR_SHAPE, "block must be 64, 128 or 256");
  if (k % block) return set_error(SDQ_ERR_SHAPE, "k=%lld is not a multiple of the block %d",
                                  (long long)k, block);
  if (levels != 2 && levels != 3) return set_error(SDQ_ERR_LEVELS, "levels=%d", levels);
  if (!(osr >= 1.0) || !(osr <= 8.0))
    return set_error(SDQ_ERR_OSR, "osr must be within [1, 8]");
  const double mf = std::nearbyint(osr * block);
  const int32_t m_up = static_cast<int32_t>(mf);
  if (m_up < block || m_up % 32)
    return set_error(SDQ_ERR_OSR, "M = round(osr*B) = %d must be a multiple of 32 and >= B", m_up);
  sdq_layout L;
  std::memset(&L, 0, sizeof(L));
  L.n = n;
  L.k = k;
  L.block = block;
  L.m_up = m_up;
  L.levels = levels;
  L.bits = levels == 2 ? 1 : 2;
  L.nb = k / block;
  L.k_up = L.nb * m_up;
  L.n_pad = (n + kPanel - 1) / kPanel * kPanel;
  L.codes_per_chunk = kChunkBytes * 8 / L.bits;
  L.n_chunks = (L.k_up + L.codes_per_chunk - 1) / L.codes_per_chunk;
  L.hadamard = SDQ_HAD_SYLVESTER;
  *out = L;
  return SDQ_OK;
}

sdq_status sdq_layout_set_packing(sdq_layout* L, int32_t packing) {
  if (!L) return set_error(SDQ_ERR_ARG, "layout is NULL");
  if (packing != SDQ_PACK_FIELDS && packing != SDQ_PACK_BASE3)
    return set_error(SDQ_ERR_ARG, "packing %d is not SDQ_PACK_FIELDS or SDQ_PACK_BASE3", packing);
  if (packing == SDQ_PACK_BASE3 && L->levels != 3)
    return set_error(SDQ_ERR_LEVELS, "base-3 packing needs ternary codes");
  sdq_layout T = *L;
  T.packing = packing;
  T.codes_per_chunk = packing == SDQ_PACK_BASE3 ? kBase3PerChunk : kChunkBytes * 8 / T.bits;
  T.n_chunks = (T.k_up + T.codes_per_chunk - 1) / T.codes_per_chunk;
  if (check_layout(&T) != SDQ_OK) return set_error(SDQ_ERR_ARG, "layout is not one produced by sdq_layout_init");
  *L = T;
  return SDQ_OK;
}

sdq_status sdq_layout_set_hadamard(sdq_layout* L, int32_t mode, const int8_t* signs) {
  if (!L) return set_error(SDQ_ERR_ARG, "layout is NULL");
  if (mode != SDQ_HAD_NONE && mode != SDQ_HAD_SYLVESTER && mode != SDQ_HAD_SIGNED)
    return set_error(SDQ_ERR_ARG, "hadamard mode %d is not SDQ_HAD_NONE, _SYLVESTER or _SIGNED", mode);
  if (!valid_block(L->block)) return set_error(SDQ_ERR_ARG, "layout is not one produced by sdq_layout_init");
  uint32_t words[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (mode == SDQ_HAD_SIGNED) {
    if (!signs) return set_error(SDQ_ERR_ARG, "the signed Hadamard needs %d signs", L->block);
    for (int t = 0; t < L->block; ++t) {
      if (signs[t] != 1 && signs[t] != -1) return set_error(SDQ_ERR_ARG, "sign %d is %d, not +-1", t, signs[t]);
      if (signs[t] < 0) words[t / 32] |= 1u << (t % 32);
    }
  }
  L->hadamard = mode;
  std::copy(words, words + 8, L->had_signs);
  return SDQ_OK;
}

size_t sdq_codes_bytes(const sdq_layout* L) {
  if (!L) return 0;
  return static_cast<size_t>(L->n_pad) * L->n_chunks * kChunkBytes;
}

double sdq_compression_ratio(const sdq_layout* L) {
  if (!L || !L->block) return 0.0;
  const double bits = L->packing == SDQ_PACK_BASE3 ? 1.6 : static_cast<double>(L->bits);
  return bits * (static_cast<double>(L->m_up) / L->block) / 16.0;
}

// Weights, activations, codes and workspaces are accessed in 16-byte vectors.
static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t sdq_quantize_workspace_bytes(const sdq_layout* L) {
  if (check_layout(L) != SDQ_OK) return 0;
  return quant_ws_layout(L, nullptr, nullptr);
}

sdq_status sdq_quantize(const float* w, const sdq_layout* L, void* codes, float* scales,
                        void* ws, size_t ws_bytes, void* stream) {
  sdq_status st = check_layout(L);
  if (st != SDQ_OK) return st;
  if (L->n > 0 && (!w || !codes || !scales))
    return set_error(SDQ_ERR_ARG, "w, codes and scales must be non-NULL");
  const size_t need = quant_ws_layout(L, nullptr, nullptr);
  if (!ws || ws_bytes < need)
    return set_error(SDQ_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  if (!aligned16(w) || !aligned16(codes) || !aligned16(ws))
    return set_error(SDQ_ERR_ARG, "w, codes and the workspace must be 16-byte aligned");
  if (L->n == 0) return SDQ_OK;
  const Tables* T = nullptr;
  st = get_tables(L, &T);
  if (st != SDQ_OK) return st;
  QuantWs qw;
  quant_ws_layout(L, &qw, ws);
  return launch_quantize(w, L, T, codes, scales, qw, static_cast<hipStream_t>(stream));
}

sdq_status sdq_quantize_check(const void* ws, void* stream) {
  if (!ws) return set_error(SDQ_ERR_ARG, "workspace is NULL");
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_error(e, "hipStreamSynchronize");
  uint32_t flag = 0;
  e = hipMemcpy(&flag, ws, sizeof(flag), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_error(e, "reading the status flag");
  if (flag) return set_error(SDQ_ERR_NONFINITE, "a weight or an upsampled sample is not finite");
  return SDQ_OK;
}

sdq_status sdq_hessian_accumulate(const float* x, int64_t m, int64_t k, double* h, void* stream) {
  if (m < 0 || k <= 0) return set_error(SDQ_ERR_ARG, "need m >= 0 and k > 0");
  if (m == 0) return SDQ_OK;
  if (!x || !h) return set_error(SDQ_ERR_ARG, "x and h must be non-NULL");
  return launch_hessian_accumulate(x, m, k, h, static_cast<hipStream_t>(stream));
}

size_t sdq_hessian_factor_workspace_bytes(int64_t k) {
  if (k <= 0 || k % 64) return 0;
  return hessian_factor_ws_bytes(k);
}

sdq_status sdq_hessian_factor(const double* h, int64_t k, double lambda, double* u, void* ws,
                              size_t ws_bytes, void* stream) {
  if (k <= 0 || k % 64) return set_error(SDQ_ERR_SHAPE, "k=%lld must be a positive multiple of 64", (long long)k);
  if (!h || !u) return set_error(SDQ_ERR_ARG, "h and u must be non-NULL");
  if (!(lambda >= 0.0) || !std::isfinite(lambda)) return set_error(SDQ_ERR_ARG, "lambda must be finite and >= 0");
  const size_t need = hessian_factor_ws_bytes(k);
  if (!ws || ws_bytes < need)
    return set_error(SDQ_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  return launch_hessian_factor(h, k, lambda, u, ws, static_cast<hipStream_t>(stream));
}

sdq_status sdq_hessian_check(const void* ws, void* stream) {
  if (!ws) return set_error(SDQ_ERR_ARG, "workspace is NULL");
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_error(e, "hipStreamSynchronize");
  int info = 0;
  e = hipMemcpy(&info, ws, sizeof(info), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_error(e, "reading the factorisation status");
  if (info) return set_error(SDQ_ERR_NOT_SPD, "H + lambda I is not positive definite in fp64");
  return SDQ_OK;
}

size_t sdq_quantize_compensated_workspace_bytes(const sdq_layout* L) {
  if (check_layout(L) != SDQ_OK) return 0;
  return comp_ws_bytes(L);
}

sdq_status sdq_quantize_compensated(const float* w, const sdq_layout* L, const double* u, int32_t update,
                                    void* codes, float* scales, void* ws, size_t ws_bytes, void* stream) {
  sdq_status st = check_layout(L);
  if (st != SDQ_OK) return st;
  if (update != SDQ_COMP_GPTQ && update != SDQ_COMP_JOINT)
    return set_error(SDQ_ERR_ARG, "update %d is not SDQ_COMP_GPTQ or SDQ_COMP_JOINT", update);
  if (L->n > 0 && (!w || !u || !codes || !scales))
    return set_error(SDQ_ERR_ARG, "w, u, codes and scales must be non-NULL");
  const size_t need = comp_ws_bytes(L);
  if (!ws || ws_bytes < need)
    return set_error(SDQ_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  if (!aligned16(w) || !aligned16(codes) || !aligned16(ws))
    return set_error(SDQ_ERR_ARG, "w, codes and the workspace must be 16-byte aligned");
  if (L->n == 0) return SDQ_OK;
  const Tables* T = nullptr;
  st = get_tables(L, &T);
  if (st != SDQ_OK) return st;
  return launch_quantize_compensated(w, L, T, u, update, codes, scales, ws, static_cast<hipStream_t>(stream));
}

// The layout a linear path reads: base-3 codes are read as stored by the
// one-row table GEMV and unpacked to 2-bit fields (into the workspace, after
// the path's own part) for every other path.
static bool needs_unpack(const sdq_layout* L, int64_t m) {
  return L->packing == SDQ_PACK_BASE3 && !(m <= 16 && decode_reads_base3(L, m));
}

static size_t path_ws_bytes(const sdq_layout* P, int64_t m) {
  return m <= 16 ? decode_ws_bytes(P, m) : prefill_ws_bytes(P, m);
}

// Workspace of a linear call over `count` linears of one layout family: the
// path's part (the expansion at offset 0), then for base-3 codes read as
// 2-bit fields each linear's unpacked copy.
static size_t group_ws_bytes(const sdq_layout* Ls, int count, int64_t m) {
  const sdq_layout* L = &Ls[0];
  if (!needs_unpack(L, m)) return path_ws_bytes(L, m);
  const sdq_layout F = fields_view(L);
  size_t off = align_up(path_ws_bytes(&F, m), 256);
  for (int j = 0; j < count; ++j) off = align_up(off + fields_codes_bytes(&Ls[j]), 256);
  return off;
}

static size_t linear_ws_bytes(const sdq_layout* L, int64_t m) { return group_ws_bytes(L, 1, m); }

size_t sdq_linear_workspace_bytes(const sdq_layout* L, int64_t m) {
  if (check_layout(L) != SDQ_OK || m < 0) return 0;
  if (m == 0) return 0;
  return linear_ws_bytes(L, m);
}

static sdq_status workspace_ok(size_t need, size_t ws_bytes, const void* ws) {
  if (!ws || ws_bytes < need)
    return set_error(SDQ_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  if (!aligned16(ws)) return set_error(SDQ_ERR_ARG, "workspace is not 16-byte aligned");
  return SDQ_OK;
}

static sdq_status linear_common(const sdq_layout* L, int64_t m, size_t ws_bytes, const void* ws) {
  sdq_status st = check_layout(L);
  if (st != SDQ_OK) return st;
  if (m < 0) return set_error(SDQ_ERR_ARG, "m < 0");
  if (m == 0 || L->n == 0) return SDQ_OK;
  if (m <= 16) {
    st = decode_supported(L);
    if (st != SDQ_OK) return st;
  }
  return workspace_ok(linear_ws_bytes(L, m), ws_bytes, ws);
}

// The expansion for layout L; `zero`: the set whose outputs the decode
// expansion zeroes for a split-K GEMV (or NULL).
static sdq_status expand_impl(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                              void* ws, const LinearSet* zero, void* stream, bool may_allocate = true) {
  if (xt != SDQ_F16 && xt != SDQ_BF16 && xt != SDQ_F32) return set_error(SDQ_ERR_ARG, "bad dtype");
  if (!x) return set_error(SDQ_ERR_ARG, "x is NULL");
  if (!aligned16(x)) return set_error(SDQ_ERR_ARG, "x is not 16-byte aligned");
  const sdq_layout F = fields_view(L);
  const sdq_layout* P = needs_unpack(L, m) ? &F : L;
  const Tables* T = nullptr;
  sdq_status st = may_allocate ? get_tables(P, &T) : find_tables(P, &T);
  if (st != SDQ_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return m <= 16 ? launch_decode_expand(x, xt, m, P, T, ws, zero, s)
                 : launch_prefill_expand(x, xt, m, P, T, ws, s);
}

// The contraction of every linear of S (layout family L) against the
// expansion in ws; base-3 codes on the paths that read 2-bit fields are
// unpacked first, each into its own part of the workspace.
static sdq_status contract_impl(int64_t m, LinearSet S, const sdq_layout* L, bool accumulate, void* ws,
                                bool y_ready, void* stream) {
  for (int j = 0; j < S.count; ++j) {
    if (!S.codes[j] || !S.scales[j] || !S.y[j]) return set_error(SDQ_ERR_ARG, "NULL pointer argument");
    if (!aligned16(S.codes[j])) return set_error(SDQ_ERR_ARG, "codes are not 16-byte aligned");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const sdq_layout F = fields_view(L);
  const sdq_layout* P = L;
  if (needs_unpack(L, m)) {
    P = &F;
    size_t off = align_up(path_ws_bytes(P, m), 256);
    for (int j = 0; j < S.count; ++j) {
      sdq_layout Lj = *L;
      Lj.n = S.n[j];
      Lj.n_pad = (S.n[j] + kPanel - 1) / kPanel * kPanel;
      uint32_t* fields = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + off);
      sdq_status st = launch_unpack_base3(S.codes[j], &Lj, fields, s);
      if (st != SDQ_OK) return st;
      S.codes[j] = fields;
      off = align_up(off + fields_codes_bytes(&Lj), 256);
    }
  }
  return m <= 16 ? launch_decode_contract(m, S, P, accumulate, ws, y_ready, s)
                 : launch_prefill_contract(m, S, P, accumulate, ws, s);
}

static LinearSet single_set(const void* codes, const float* scales, const sdq_layout* L, float* y) {
  LinearSet S;
  S.count = 1;
  S.codes[0] = codes;
  S.scales[0] = scales;
  S.y[0] = y;
  S.n[0] = L->n;
  return S;
}

sdq_status sdq_expand_activations(const void* x, sdq_dtype xt, int64_t m, const sdq_layout* L,
                                  void* ws, size_t ws_bytes, void* stream) {
  sdq_status st = linear_common(L, m, ws_bytes, ws);
  if (st != SDQ_OK || m == 0 || L->n == 0) return st;
  return expand_impl(x, xt, m, L, ws, nullptr, stream);
}

sdq_status sdq_linear_expanded(int64_t m, const void* codes, const float* scales,
                               const sdq_layout* L, float* y, int32_t accumulate, void* ws,
                               size_t ws_bytes, void* stream) {
  sdq_status st = linear_common(L, m, ws_bytes, ws);
  if (st != SDQ_OK || m == 0 || L->n == 0) return st;
  return contract_impl(m, single_set(codes, scales, L, y), L, accumulate != 0, ws, false, stream);
}

// Argument checks of sdq_linear that precede the workspace check.
static sdq_status linear_args(const void* x, sdq_dtype xt, int64_t m, const void* codes, const float* scales,
                              const sdq_layout* L, const float* y) {
  sdq_status st = check_layout(L);
  if (st != SDQ_OK) return st;
  if (m < 0) return set_error(SDQ_ERR_ARG, "m < 0");
  if (xt != SDQ_F16 && xt != SDQ_BF16 && xt != SDQ_F32) return set_error(SDQ_ERR_ARG, "bad dtype");
  if (m == 0 || L->n == 0) return SDQ_OK;
  if (!x || !codes || !scales || !y) return set_error(SDQ_ERR_ARG, "NULL pointer argument");
  if (!aligned16(x) || !aligned16(codes)) return set_error(SDQ_ERR_ARG, "x and codes must be 16-byte aligned");
  return SDQ_OK;
}

// Expansion then contraction of a set on one workspace (sdq_linear and
// sdq_linear_group).  Decode: the expansion also zeroes y when the GEMV
// will add into it.
static sdq_status run_set(const void* x, sdq_dtype xt, int64_t m, const LinearSet& S, const sdq_layout* L,
                          int32_t accumulate, void* ws, void* stream, bool may_allocate) {
  const sdq_layout F = fields_view(L);
  const sdq_layout* P = needs_unpack(L, m) ? &F : L;
  const bool zero_in_expand = !accumulate && m <= 16 && decode_needs_zero_y(P, m, set_panels(S));
  sdq_status st = expand_impl(x, xt, m, L, ws, zero_in_expand ? &S : nullptr, stream, may_allocate);
  if (st != SDQ_OK) return st;
  return contract_impl(m, S, L, accumulate != 0, ws, true, stream);
}

}  // extern "C"

sdq_status sdq::linear_impl(const void* x, sdq_dtype xt, int64_t m, const void* codes, const float* scales,
                            const sdq_layout* L, float* y, int32_t accumulate, void* ws, size_t ws_bytes,
                            void* stream, bool may_allocate) {
  sdq_status st = linear_args(x, xt, m, codes, scales, L, y);
  if (st != SDQ_OK || m == 0 || L->n == 0) return st;
  st = linear_common(L, m, ws_bytes, ws);
  if (st != SDQ_OK) return st;
  return run_set(x, xt, m, single_set(codes, scales, L, y), L, accumulate, ws, stream, may_allocate);
}

size_t sdq::linear_ws_need(const sdq_layout* L, int64_t m) {
  if (check_layout(L) != SDQ_OK || m <= 0) return 0;
  return linear_ws_bytes(L, m);
}

extern "C" {

sdq_status sdq_linear(const void* x, sdq_dtype xt, int64_t m, const void* codes,
                      const float* scales, const sdq_layout* L, float* y, int32_t accumulate,
                      void* ws, size_t ws_bytes, void* stream) {
  return linear_impl(x, xt, m, codes, scales, L, y, accumulate, ws, ws_bytes, stream, true);
}

// Layouts of one group: valid, and equal in everything the expansion and the
// code geometry depend on (all but the row count).
static sdq_status check_group(const sdq_layout* Ls, int32_t count) {
  if (count < 1 || count > kMaxGroup)
    return set_error(SDQ_ERR_ARG, "count=%d: a group holds 1 to %d linears", count, kMaxGroup);
  if (!Ls) return set_error(SDQ_ERR_ARG, "layouts is NULL");
  for (int j = 0; j < count; ++j) {
    sdq_status st = check_layout(&Ls[j]);
    if (st != SDQ_OK) return st;
    const sdq_layout& a = Ls[0];
    const sdq_layout& b = Ls[j];
    if (a.k != b.k || a.block != b.block || a.m_up != b.m_up || a.levels != b.levels ||
        a.hadamard != b.hadamard || a.packing != b.packing ||
        !std::equal(a.had_signs, a.had_signs + 8, b.had_signs))
      return set_error(SDQ_ERR_ARG, "linear %d differs from linear 0 in k, block, M, levels, Had or packing", j);
  }
  return SDQ_OK;
}

size_t sdq_linear_group_workspace_bytes(const sdq_layout* layouts, int32_t count, int64_t m) {
  if (check_group(layouts, count) != SDQ_OK || m <= 0) return 0;
  return group_ws_bytes(layouts, count, m);
}

// The set of a group call (empty linears left out) after its checks.
static sdq_status group_set(int64_t m, int32_t count, const void* const* codes, const float* const* scales,
                            const sdq_layout* layouts, float* const* y, size_t ws_bytes, const void* ws,
                            LinearSet* S) {
  sdq_status st = check_group(layouts, count);
  if (st != SDQ_OK) return st;
  if (m < 0) return set_error(SDQ_ERR_ARG, "m < 0");
  if (!codes || !scales || !y) return set_error(SDQ_ERR_ARG, "NULL pointer array");
  for (int j = 0; j < count; ++j) {
    if (layouts[j].n == 0) continue;            // nothing to compute for an empty linear
    S->codes[S->count] = codes[j];
    S->scales[S->count] = scales[j];
    S->y[S->count] = y[j];
    S->n[S->count] = layouts[j].n;
    ++S->count;
  }
  if (m == 0 || S->count == 0) return SDQ_OK;
  if (m <= 16) {
    st = decode_supported(&layouts[0]);
    if (st != SDQ_OK) return st;
  }
  return workspace_ok(group_ws_bytes(layouts, count, m), ws_bytes, ws);
}

sdq_status sdq_linear_group(const void* x, sdq_dtype xt, int64_t m, int32_t count, const void* const* codes,
                            const float* const* scales, const sdq_layout* layouts, float* const* y,
                            int32_t accumulate, void* ws, size_t ws_bytes, void* stream) {
  if (xt != SDQ_F16 && xt != SDQ_BF16 && xt != SDQ_F32) return set_error(SDQ_ERR_ARG, "bad dtype");
  LinearSet S;
  sdq_status st = group_set(m, count, codes, scales, layouts, y, ws_bytes, ws, &S);
  if (st != SDQ_OK || m == 0 || S.count == 0) return st;
  if (!x) return set_error(SDQ_ERR_ARG, "x is NULL");
  return run_set(x, xt, m, S, &layouts[0], accumulate, ws, stream, true);
}

sdq_status sdq_linear_group_expanded(int64_t m, int32_t count, const void* const* codes,
                                     const float* const* scales, const sdq_layout* layouts, float* const* y,
                                     int32_t accumulate, void* ws, size_t ws_bytes, void* stream) {
  LinearSet S;
  sdq_status st = group_set(m, count, codes, scales, layouts, y, ws_bytes, ws, &S);
  if (st != SDQ_OK || m == 0 || S.count == 0) return st;
  return contract_impl(m, S, &layouts[0], accumulate != 0, ws, false, stream);
}

// ---------------------------------------------------------------------------
// MultiOSR (Section 3.4), host only.
// ---------------------------------------------------------------------------
static double weighted_clip(double scale, const std::vector<double>& sc,
                            const std::vector<double>& wt, double lo, double hi) {
  double tot = 0.0;
  for (size_t i = 0; i < sc.size(); ++i) {
    const double val = std::isinf(sc[i]) ? hi : std::min(std::max(scale * sc[i], lo), hi);
    tot += wt[i] * val;
  }
  return tot;
}

static std::vector<double> allocate(const std::vector<double>& sc, const std::vector<double>& wt,
                                    double target, double lo, double hi) {
  const size_t n = sc.size();
  if (target <= lo) return std::vector<double>(n, lo);
  if (target >= hi) return std::vector<double>(n, hi);
  double wsum = 0.0;
  for (double w : wt) wsum += w;
  double min_finite = INFINITY;
  for (double s : sc)
    if (!std::isinf(s)) min_finite = std::min(min_finite, s);
  if (std::isinf(min_finite)) return std::vector<double>(n, hi);
  double c_lo = 0.0, c_hi = hi / min_finite;
  const double goal = target * wsum;
  for (int it = 0; it < 200; ++it) {
    const double mid = 0.5 * (c_lo + c_hi);
    if (weighted_clip(mid, sc, wt, lo, hi) < goal) c_lo = mid;
    else c_hi = mid;
  }
  std::vector<double> out(n);
  for (size_t i = 0; i < n; ++i)
    out[i] = std::isinf(sc[i]) ? hi : std::min(std::max(c_hi * sc[i], lo), hi);
  return out;
}

sdq_status sdq_multiosr(const double* var, const int64_t* np, const int32_t* layer, int64_t count,
                        double target, double lo, double hi, double grid, double* out) {
  if (count < 0) return set_error(SDQ_ERR_ARG, "count < 0");
  if (!(lo > 0) || !(lo <= target) || !(target <= hi) || !(grid > 0))
    return set_error(SDQ_ERR_ARG, "need 0 < lo <= target <= hi and grid > 0");
  if (count == 0) return SDQ_OK;
  if (!var || !np || !layer || !out) return set_error(SDQ_ERR_ARG, "NULL pointer argument");
  for (int64_t j = 0; j < count; ++j)
    if (np[j] <= 0) return set_error(SDQ_ERR_ARG, "parameter count of linear %lld is <= 0", (long long)j);
  // Layer level: score 1 / (parameter-weighted variance).
  std::vector<int32_t> layers(layer, layer + count);
  std::sort(layers.begin(), layers.end());
  layers.erase(std::unique(layers.begin(), layers.end()), layers.end());
  std::vector<double> lay_sc, lay_n;
  std::vector<std::vector<int64_t>> members(layers.size());
  for (size_t l = 0; l < layers.size(); ++l) {
    int64_t n_l = 0;
    double acc = 0.0;
    for (int64_t j = 0; j < count; ++j)
      if (layer[j] == layers[l]) {
        members[l].push_back(j);
        n_l += np[j];
        acc += static_cast<double>(np[j]) * var[j];
      }
    const double pooled = acc / static_cast<double>(n_l);
    lay_n.push_back(static_cast<double>(n_l));
    lay_sc.push_back(pooled <= 0 ? INFINITY : 1.0 / pooled);
  }
  const std::vector<double> lay_osr = allocate(lay_sc, lay_n, target, lo, hi);
  // Linear level: score n_j / var_j inside each layer.
  std::vector<double> cont(count);
  for (size_t l = 0; l < layers.size(); ++l) {
    std::vector<double> sc, wt;
    for (int64_t j : members[l]) {
      sc.push_back(var[j] <= 0 ? INFINITY : static_cast<double>(np[j]) / var[j]);
      wt.push_back(static_cast<double>(np[j]));
    }
    const std::vector<double> v = allocate(sc, wt, lay_osr[l], lo, hi);
    for (size_t i = 0; i < members[l].size(); ++i) cont[members[l][i]] = v[i];
  }
  // Snap: floor to the grid, then add steps by decreasing remainder within the budget.
  const int64_t k_lo = static_cast<int64_t>(std::ceil(lo / grid - 1e-9));
  const int64_t k_hi = static_cast<int64_t>(std::floor(hi / grid + 1e-9));
  std::vector<int64_t> ks(count);
  std::vector<double> rem(count);
  int64_t ntot = 0, used = 0;
  for (int64_t j = 0; j < count; ++j) {
    const double q = cont[j] / grid;
    int64_t k = static_cast<int64_t>(std::floor(q + 1e-9));
    k = std::min(std::max(k, k_lo), k_hi);
    ks[j] = k;
    rem[j] = q - static_cast<double>(k);
    ntot += np[j];
    used += np[j] * k;
  }
  const double budget = target / grid * static_cast<double>(ntot);
  std::vector<int64_t> order(count);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) {
    if (rem[a] != rem[b]) return rem[a] > rem[b];
    return a < b;
  });
  for (int64_t j : order) {
    if (ks[j] + 1 <= k_hi && static_cast<double>(used + np[j]) <= budget) {
      ks[j] += 1;
      used += np[j];
    }
  }
  for (int64_t j = 0; j < count; ++j) out[j] = static_cast<double>(ks[j]) * grid;
  return SDQ_OK;
}

sdq_status sdq_unpack_codes(const sdq_layout* L, const void* codes_host, int8_t* out) {
  sdq_status st = check_layout(L);
  if (st != SDQ_OK) return st;
  if (L->n > 0 && (!codes_host || !out)) return set_error(SDQ_ERR_ARG, "NULL pointer argument");
  if (L->packing == SDQ_PACK_BASE3) {
    const uint8_t* bytes = static_cast<const uint8_t*>(codes_host);
    for (int64_t r = 0; r < L->n; ++r)
      for (int64_t j = 0; j < L->k_up; ++j) {
        const int64_t c = j / kBase3PerChunk, q = j % kBase3PerChunk;
        const int64_t chunk = ((r / kPanel) * L->n_chunks + c) * kPanel + (r % kPanel);
        int v = 243 * bytes[chunk * kChunkBytes + q / 5] / 256;
        for (int i = q % 5; i < 4; ++i) v /= 3;
        out[r * L->k_up + j] = static_cast<int8_t>(v % 3 - 1);
      }
    return SDQ_OK;
  }
  const uint32_t* words = static_cast<const uint32_t*>(codes_host);
  const int bits = L->bits;
  const int per_word = 32 / bits;
  const uint32_t mask = (1u << bits) - 1u;
  for (int64_t r = 0; r < L->n; ++r) {
    for (int64_t j = 0; j < L->k_up; ++j) {
      const int64_t c = j / L->codes_per_chunk;
      const int64_t q = j % L->codes_per_chunk;
      const int64_t chunk = ((r / kPanel) * L->n_chunks + c) * kPanel + (r % kPanel);
      const uint32_t wv = words[chunk * 4 + q / per_word];
      const uint32_t f = (wv >> (bits * (q % per_word))) & mask;
      int8_t v;
      if (bits == 1) v = f ? 1 : -1;
      else v = f == 1 ? 1 : (f == 3 ? -1 : 0);
      out[r * L->k_up + j] = v;
    }
  }
  return SDQ_OK;
}

sdq_status sdq_upsample_table(int32_t block, int32_t m_up, float* out) {
  if (!out) return set_error(SDQ_ERR_ARG, "out is NULL");
  if (!valid_block(block)) return set_error(SDQ_ERR_SHAPE, "block must be 64, 128 or 256");
  if (m_up < block || m_up % 32 || m_up > 8 * block) return set_error(SDQ_ERR_OSR, "bad M=%d", m_up);
  const int64_t bm = static_cast<int64_t>(block) * m_up;
  for (int64_t p = 0; p < bm; ++p) out[p] = static_cast<float>(upsample_kernel(p, block, m_up));
  return SDQ_OK;
}

sdq_status sdq_prepare(int32_t block, int32_t m_up) {
  if (!valid_block(block)) return set_error(SDQ_ERR_SHAPE, "block must be 64, 128 or 256");
  if (m_up < block || m_up % 32 || m_up > 8 * block) return set_error(SDQ_ERR_OSR, "bad M=%d", m_up);
  const Tables* T = nullptr;
  return get_tables_for(block, m_up, SDQ_HAD_SYLVESTER, SignWords{}, &T);
}

sdq_status sdq_prepare_layout(const sdq_layout* L) {
  sdq_status st = check_layout(L);
  if (st != SDQ_OK) return st;
  const Tables* T = nullptr;
  return get_tables(L, &T);
}

void sdq_release_tables(void) {
  std::lock_guard<std::mutex> lock(g_tables_mutex);
  for (auto& kv : g_tables) {
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(std::get<0>(kv.first));
    if (kv.second.unz) (void)hipFree(kv.second.unz);
    if (kv.second.edec) (void)hipFree(kv.second.edec);
    if (kv.second.et_hi) (void)hipFree(kv.second.et_hi);
    if (kv.second.et_lo) (void)hipFree(kv.second.et_lo);
    if (kv.second.e64) (void)hipFree(kv.second.e64);
    (void)hipSetDevice(cur);
  }
  g_tables.clear();
}

size_t sdq_moments_workspace_bytes(int64_t count) { return count < 0 ? 0 : moments_ws_bytes(count); }

sdq_status sdq_weight_moments(const float* w, int64_t count, double* out, void* ws, size_t ws_bytes,
                              void* stream) {
  if (count <= 0 || !w || !out) return set_error(SDQ_ERR_ARG, "need count > 0 and non-NULL pointers");
  const size_t need = moments_ws_bytes(count);
  if (!ws || ws_bytes < need)
    return set_error(SDQ_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  return launch_moments(w, count, out, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

}  // extern "C"
