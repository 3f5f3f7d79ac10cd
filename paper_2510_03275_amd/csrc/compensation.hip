// Block compensation of Algorithm 1 (the block loop), fp64 on the device.
//
//   hessian  H += 2 X^T X for calibration activations X (m x K).
//   factor   U = Cholesky((H + lambda I)^-1)^T, upper, U^T U = (H + lambda I)^-1.
//            Computed without forming the inverse: with J the index reversal,
//            J (H + lambda I) J = L L^T (blocked Cholesky, 64-column panels)
//            and U = J L^-1 J (blocked triangular inverse), because
//            (J L^-1 J)^T (J L^-1 J) = J (L L^T)^-1 J = (H + lambda I)^-1.
//   encode   the weight's row scales come from the uncompensated W (the plain
//            encoder); W is then carried in fp64 and walked in blocks of B
//            columns: block b is rounded to fp32 and encoded with those
//            scales (the same rotate / upsample / scan kernels), its
//            reconstruction Q_b = (s * C_b) E^T (E = Had D^T, the table of the
//            activation expansion, in fp64) gives the error E_b = W_b - Q_b, and
//            the later columns are corrected with GPTQ's block step without its
//            column-wise part, W_F -= E_b diag(U_QQ)^-1 U_QF (each column's
//            error divided by its pivot), or optionally with the
//            optimal-brain-surgeon correction of the jointly quantized block,
//            W_F -= E_b U_QQ^-1 U_QF.
//
// All of it is dense fp64 linear algebra: one GEMM on the fp64 matrix cores
// with general strides (64 x 64 tile per workgroup, 16-deep k slices through
// LDS) serves the Hessian, the panel solves, the trailing updates, the
// triangular inverses and the block corrections.  The 64 x 64 diagonal
// blocks of the Cholesky factor are factored and inverted in registers by one
// workgroup, fused into the trailing update that produces them; another small
// kernel inverts given triangular 64-blocks in LDS.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "sdq_internal.h"

namespace sdq {
namespace {

constexpr int kT = 64;     // factorisation panel / GEMM tile
constexpr int kTK = 16;    // GEMM k step
constexpr int kStage = kT * kTK / 256;   // operand elements staged per thread and k step

// Cholesky factor and inverse of one 64 x 64 block in place: the lower part
// of A (row stride lda, unit column stride) is read, A = L L^T is written back
// with the upper part zeroed and X = L^-1 (lower) is written.  Symmetric
// elimination without square roots: step j takes column j of the reduced
// matrix (pivot d_j), forms the multipliers m_i = c_i / d_j of the rows below
// it and subtracts m_i times row j from row i, in the reduced matrix and in a
// copy of the identity, which becomes L'^-1 for the unit lower factor of
// A = L' D L'^T.  Then column j of L is c / sqrt(d_j) and L^-1 = D^-1/2 L'^-1
// (row i divided by sqrt(d_i)).  Thread t keeps a 4 x 4 tile of the reduced
// matrix and of the inverse in registers (rows 4 (t / 16) .., columns
// 4 (t % 16) ..; a finished column stays in place).  Per step, the owners of
// the next column and of the next row of the inverse update those first and
// publish them in a two-slot LDS ring, with the next-but-one diagonal entry;
// from that entry every thread forms the next pivot and its reciprocal while
// the rest of the tile is updated, so only a multiply and an FMA lie between
// two barriers on the column-to-column path (one barrier per column).  Upper
// entries of the tiles are updated too and never read.  A pivot that is not
// positive sets *info and is taken as 1.  Needs 256 threads and 322 doubles of
// LDS at lds.
__device__ __forceinline__ void chol64_tile(double* A, int64_t lda, double* X, int64_t ldx, int* info,
                                            double* lds) {
  double(*ct)[kT] = reinterpret_cast<double(*)[kT]>(lds);            // column j in slot j % 2
  double(*xr)[kT] = reinterpret_cast<double(*)[kT]>(lds + 2 * kT);   // row j of L'^-1, slot j % 2
  double* ev = lds + 4 * kT;                                          // diagonal entry j in slot j % 2
  double* dv = lds + 4 * kT + 2;                                      // pivots
  const int tid = threadIdx.x;
  const int ti = tid / 16, tk = tid % 16;
  const int i0 = 4 * ti, k0 = 4 * tk;
  double a[4][4], x[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      a[r][c] = k0 + c <= i0 + r ? A[(i0 + r) * lda + k0 + c] : 0.0;
      x[r][c] = i0 + r == k0 + c ? 1.0 : 0.0;
    }
  }
  if (tk == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) ct[0][i0 + r] = a[r][0];
  }
  if (ti == 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) xr[0][k0 + c] = x[0][c];
  }
  if (tid == 0) ev[1] = a[1][1];
  __syncthreads();
  double d = ct[0][0];
  if (!(d > 0.0)) {
    if (tid == 0) info[0] = 1;
    d = 1.0;
  }
  if (tid == 0) dv[0] = d;
  double rd = 1.0 / d;
  for (int jb = 0; jb < kT; jb += 4) {
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int j = jb + jj, sl = jj & 1, sn = sl ^ 1;
      const int jn = j + 1, cn = (jj + 1) & 3, c2 = (jj + 2) & 3;
      // All of the step's LDS reads first, unconditionally (a select after
      // the load keeps them out of branches).
      const double2 cr0 = *reinterpret_cast<const double2*>(&ct[sl][i0]);
      const double2 cr1 = *reinterpret_cast<const double2*>(&ct[sl][i0 + 2]);
      const double2 cc0 = *reinterpret_cast<const double2*>(&ct[sl][k0]);
      const double2 cc1 = *reinterpret_cast<const double2*>(&ct[sl][k0 + 2]);
      const double2 xx0 = *reinterpret_cast<const double2*>(&xr[sl][k0]);
      const double2 xx1 = *reinterpret_cast<const double2*>(&xr[sl][k0 + 2]);
      const double cj = ct[sl][jn < kT ? jn : j];
      const double en = ev[sn];
      const double crv[4] = {cr0.x, cr0.y, cr1.x, cr1.y};
      const double ccv[4] = {cc0.x, cc0.y, cc1.x, cc1.y};
      double m[4], ck[4];
      const double xk[4] = {xx0.x, xx0.y, xx1.x, xx1.y};
#pragma unroll
      for (int r = 0; r < 4; ++r) m[r] = crv[r] * (i0 + r > j ? rd : 0.0);   // (entries above j are finite)
#pragma unroll
      for (int c = 0; c < 4; ++c) ck[c] = k0 + c > j ? ccv[c] : 0.0;
      if (jn < kT) {
        if (tk == jn / 4) {
#pragma unroll
          for (int r = 0; r < 4; ++r) ct[sn][i0 + r] = a[r][cn] - m[r] * ck[cn];
        }
        if (ti == jn / 4) {
#pragma unroll
          for (int c = 0; c < 4; ++c) xr[sn][k0 + c] = x[cn][c] - m[cn] * xk[c];
        }
        if (jn + 1 < kT && ti == (jn + 1) / 4 && tk == (jn + 1) / 4) ev[sl] = a[c2][c2] - m[c2] * ck[c2];
        // next pivot: entry (j + 1, j + 1) after this step's update
        double dn = en - (cj * rd) * cj;
        if (!(dn > 0.0)) {
          if (tid == 0) info[0] = 1;
          dn = 1.0;
        }
        if (tid == 0) dv[jn] = dn;
        rd = 1.0 / dn;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          a[r][c] -= m[r] * ck[c];
          x[r][c] -= m[r] * xk[c];
        }
      }
      __syncthreads();
    }
  }
  double* sq = ct[0];   // square roots of the pivots (the ring is free now)
  if (tid < kT) sq[tid] = sqrt(dv[tid]);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i = i0 + r, k = k0 + c;
      A[i * lda + k] = k < i ? a[r][c] / sq[k] : (k == i ? sq[i] : 0.0);
      X[i * ldx + k] = k <= i ? x[r][c] / sq[i] : 0.0;
    }
  }
}

__global__ __launch_bounds__(256) void chol64_kernel(double* A, int64_t lda, double* X, int64_t ldx,
                                                     int* info) {
  __shared__ double lds[4 * kT + 2 + kT];
  chol64_tile(A, lda, X, ldx, info, lds);
}

// C = beta C + alpha A B; element (i, p) of A at A[i * rsa + p * csa], likewise
// B and C; blockIdx.z selects a batch (strides bsa, bsb, bsc).  lower_only = 1
// skips tiles strictly above the diagonal of C; lower_only = 2 (a symmetric
// product, M = N) skips them too but also updates the transposed position of
// every tile below the diagonal, so both triangles are written.  beta == 0
// never reads C.  A and B
// may overlap C only where every output tile depends on the same rows of A
// alone (an in-place panel solve with N <= 64): a workgroup reads all of its
// operands before it writes.
//
// fp64 matrix cores: a 64 x 64 tile per workgroup, four waves in a 2 x 2 grid
// of 32 x 32 (four v_mfma_f64_16x16x4f64 accumulators each).  Operands go
// through LDS in 16-deep k slices (converted to fp64 on the way), the next
// slice loaded into registers while the current one is multiplied.  Lane
// layout of the instruction: lane l supplies A[l % 16][l / 16] and
// B[l / 16][l % 16] and receives D[l / 16 + 4 v][l % 16] in item v.
typedef double double4_t __attribute__((ext_vector_type(4)));

template <typename TA, typename TB, bool kChol = false>
__global__ __launch_bounds__(256) void gemm64_kernel(
    int64_t M, int64_t N, int64_t K, double alpha, const TA* A, int64_t rsa, int64_t csa,
    int64_t bsa, const TB* B, int64_t rsb, int64_t csb, int64_t bsb, double beta, double* C,
    int64_t rsc, int64_t csc, int64_t bsc, int lower_only, double* cx, int64_t ldx, int* info) {
  __shared__ double As[kTK][kT + 2];
  __shared__ double Bs[kTK][kT + 2];
  const int tid = threadIdx.x;
  const int lane = tid % 64, wave = tid / 64;
  const int wr = wave / 2, wc = wave % 2;
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * kT;
  const int64_t j0 = static_cast<int64_t>(blockIdx.x) * kT;
  if (lower_only && i0 + kT - 1 < j0) return;
  A += static_cast<int64_t>(blockIdx.z) * bsa;
  B += static_cast<int64_t>(blockIdx.z) * bsb;
  C += static_cast<int64_t>(blockIdx.z) * bsc;
  // Staging: element e = tid + 256 q of the slice, consecutive threads along
  // the operand's contiguous index.
  const bool a_pfast = csa == 1;
  const bool b_jfast = csb == 1;
  int aii[kStage], app[kStage], bjj[kStage], bpp[kStage];
#pragma unroll
  for (int q = 0; q < kStage; ++q) {
    const int e = tid + 256 * q;
    aii[q] = a_pfast ? e / kTK : e % kT;
    app[q] = a_pfast ? e % kTK : e / kT;
    bjj[q] = b_jfast ? e % kT : e / kTK;
    bpp[q] = b_jfast ? e / kT : e % kTK;
  }
  TA ra[kStage];
  TB rb[kStage];
  auto load = [&](int64_t p0) {
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
      const int64_t gi = i0 + aii[q], gp = p0 + app[q];
      ra[q] = gi < M && gp < K ? A[gi * rsa + gp * csa] : TA(0);
      const int64_t gj = j0 + bjj[q], gq = p0 + bpp[q];
      rb[q] = gj < N && gq < K ? B[gq * rsb + gj * csb] : TB(0);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int q = 0; q < kStage; ++q) {
      As[app[q]][aii[q]] = static_cast<double>(ra[q]);
      Bs[bpp[q]][bjj[q]] = static_cast<double>(rb[q]);
    }
  };
  double4_t acc[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c) acc[r][c] = double4_t{0.0, 0.0, 0.0, 0.0};
  const int lr = lane % 16, lk = lane / 16;
  load(0);
  store();
  __syncthreads();
  for (int64_t p0 = 0; p0 < K; p0 += kTK) {
    const bool more = p0 + kTK < K;
    if (more) load(p0 + kTK);
#pragma unroll
    for (int kk = 0; kk < kTK / 4; ++kk) {
      double a[2], b[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) a[r] = As[4 * kk + lk][32 * wr + 16 * r + lr];
#pragma unroll
      for (int c = 0; c < 2; ++c) b[c] = Bs[4 * kk + lk][32 * wc + 16 * c + lr];
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[r][c] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[r], b[c], acc[r][c], 0, 0, 0);
    }
    __syncthreads();
    if (more) {
      store();
      __syncthreads();
    }
  }
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t gi = i0 + 32 * wr + 16 * r + lk + 4 * v, gj = j0 + 32 * wc + 16 * c + lr;
        if (gi < M && gj < N) {
          double* cp = C + gi * rsc + gj * csc;
          double val = alpha * acc[r][c][v];
          if (beta != 0.0) val += beta * *cp;
          *cp = val;
          if (lower_only == 2 && i0 > j0) {
            double* mp = C + gj * rsc + gi * csc;
            double mv = alpha * acc[r][c][v];
            if (beta != 0.0) mv += beta * *mp;
            *mp = mv;
          }
        }
      }
  if constexpr (kChol) {
    // The first tile goes on to its Cholesky factor and inverse (the tile's
    // stores above are visible to the whole workgroup after the barrier).
    if (blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0) {
      __syncthreads();
      chol64_tile(C, rsc, cx, ldx, info, &As[0][0]);
    }
  }
}

// Inverse X = L^-1 of lower-triangular 64 x 64 diagonal blocks, one per
// workgroup (grid x: blocks along a diagonal, stride sa1 / sx1; grid y:
// batches, stride sa2 / sx2), in three levels: the four 16 x 16 diagonal
// blocks by forward substitution (one column per thread), then pairs of
// diagonal blocks are joined as X21 = -X22 (L21 X11), 16 -> 32 and 32 -> 64,
// every output of a product on its own thread.
__global__ __launch_bounds__(256) void trinv64_kernel(const double* A, int64_t lda, int64_t sa1, int64_t sa2,
                                                      double* X, int64_t ldx, int64_t sx1, int64_t sx2) {
  __shared__ double a[kT][kT + 1];
  __shared__ double x[kT][kT + 1];
  A += blockIdx.x * sa1 + blockIdx.y * sa2;
  X += blockIdx.x * sx1 + blockIdx.y * sx2;
  const int tid = threadIdx.x;
  for (int e = tid; e < kT * kT; e += 256) {
    const int i = e / kT, k = e % kT;
    a[i][k] = k <= i ? A[i * lda + k] : 0.0;
  }
  __syncthreads();
  __shared__ double rd[kT];          // 1 / L[i][i]
  __shared__ double tt[32 * 32];     // L21 X11 of the current level
  if (tid < kT) rd[tid] = 1.0 / a[tid][tid];
  for (int e = tid; e < kT * kT; e += 256) x[e / kT][e % kT] = 0.0;
  __syncthreads();
  if (tid < kT) {
    const int o = 16 * (tid / 16), c = tid % 16;
    for (int i = c; i < 16; ++i) {
      double s = i == c ? 1.0 : 0.0;
      for (int k = c; k < i; ++k) s -= a[o + i][o + k] * x[o + k][o + c];
      x[o + i][o + c] = s * rd[o + i];
    }
  }
  __syncthreads();
  for (int b = 16; b < kT; b *= 2) {
    const int pairs = kT / (2 * b);
    for (int e = tid; e < pairs * b * b; e += 256) {
      const int pr = e / (b * b), i = (e / b) % b, j = e % b, r = 2 * b * pr;
      double s = 0.0;
      for (int k = j; k < b; ++k) s += a[r + b + i][r + k] * x[r + k][r + j];
      tt[(pr * b + i) * b + j] = s;
    }
    __syncthreads();
    for (int e = tid; e < pairs * b * b; e += 256) {
      const int pr = e / (b * b), i = (e / b) % b, j = e % b, r = 2 * b * pr;
      double s = 0.0;
      for (int k = 0; k <= i; ++k) s += x[r + b + i][r + b + k] * tt[(pr * b + k) * b + j];
      x[r + b + i][r + j] = -s;
    }
    __syncthreads();
  }
  __syncthreads();
  for (int e = tid; e < kT * kT; e += 256) {
    const int i = e / kT, k = e % kT;
    X[i * ldx + k] = x[i][k];
  }
}

// dst[i][j] = src[n-1-i][n-1-j] (+ lam on the diagonal) where kept (i >= j
// for keep_lower, else j >= i), 0 elsewhere; grid y selects a batch.
__global__ void reverse_tri_kernel(const double* __restrict__ src, int64_t lds, int64_t ss,
                                   int64_t n, double* __restrict__ dst, int64_t ldd, int64_t sd,
                                   int keep_lower, double lam) {
  src += blockIdx.y * ss;
  dst += blockIdx.y * sd;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < n * n;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / n, j = e % n;
    const bool keep = keep_lower ? i >= j : j >= i;
    dst[i * ldd + j] = keep ? src[(n - 1 - i) * lds + (n - 1 - j)] + (i == j ? lam : 0.0) : 0.0;
  }
}

__global__ void fill_f64_kernel(double* __restrict__ p, int64_t count, double v) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = v;
}

__global__ void clear_info_kernel(int* info) { if (threadIdx.x == 0) info[0] = 0; }

__global__ void widen_kernel(const float* __restrict__ w, int64_t count, double* __restrict__ w64) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    w64[i] = static_cast<double>(w[i]);
}

// Block column col0 .. col0 + B - 1 of W64 (n x k): rounded to fp32 into wblk
// (n x B, the encoder's input) and copied into ebuf (n x B, fp64).
__global__ void extract_block_kernel(const double* __restrict__ w64, int64_t n, int64_t k, int B,
                                     int64_t col0, float* __restrict__ wblk, double* __restrict__ ebuf) {
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < n * B;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t r = e / B, t = e % B;
    const double v = w64[r * k + col0 + t];
    wblk[e] = static_cast<float>(v);
    ebuf[e] = v;
  }
}

// cb[r][m] = s_r * code(r, j0 + m) (n x M, fp64) from the packed format.
__global__ void unpack_scaled_kernel(const uint32_t* __restrict__ codes, const float* __restrict__ scales,
                                     int64_t n, int64_t n_chunks, int cpc, int bits, int64_t j0,
                                     int m_up, double* __restrict__ cb) {
  const int per_word = 32 / bits;
  for (int64_t e = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; e < n * m_up;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t r = e / m_up;
    const int64_t j = j0 + e % m_up;
    const int64_t c = j / cpc;
    const int q = static_cast<int>(j % cpc);
    const uint32_t word = codes[(((r / kPanel) * n_chunks + c) * kPanel + r % kPanel) * 4 + q / per_word];
    const uint32_t f = (word >> (bits * (q % per_word))) & ((1u << bits) - 1u);
    const double code = bits == 1 ? (f ? 1.0 : -1.0) : (f == 1u ? 1.0 : (f == 3u ? -1.0 : 0.0));
    cb[e] = static_cast<double>(scales[r]) * code;
  }
}

// g[r][t] = e[r][t] / u[c0 + t][c0 + t] (n x B): the block error of every
// column divided by that column's pivot, an IEEE division per element.
__global__ void divide_by_pivots_kernel(const double* __restrict__ e, const double* __restrict__ u,
                                        int64_t k, int64_t c0, int64_t n, int B, double* __restrict__ g) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n * B;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t t = c0 + i % B;
    g[i] = e[i] / u[t * k + t];
  }
}

unsigned grid1(int64_t count) {
  return static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 8192));
}

template <typename TA, typename TB>
void gemm64(int64_t M, int64_t N, int64_t K, double alpha, const TA* A, int64_t rsa, int64_t csa,
            const TB* B, int64_t rsb, int64_t csb, double beta, double* C, int64_t rsc, int64_t csc,
            hipStream_t stream, int lower_only = 0, int batch = 1, int64_t bsa = 0, int64_t bsb = 0,
            int64_t bsc = 0) {
  if (M <= 0 || N <= 0) return;
  const dim3 grid(static_cast<unsigned>((N + kT - 1) / kT), static_cast<unsigned>((M + kT - 1) / kT),
                  static_cast<unsigned>(batch));
  gemm64_kernel<TA, TB><<<grid, dim3(256), 0, stream>>>(M, N, K, alpha, A, rsa, csa, bsa, B, rsb, csb,
                                                        bsb, beta, C, rsc, csc, bsc, lower_only, nullptr, 0,
                                                        nullptr);
}

// Trailing update of a right-looking Cholesky step, C -= P P^T on the tiles
// on or below the diagonal (P: n x 64, row stride ld; C: n x n, row stride
// ld), whose first tile then factors and inverts the next diagonal block
// (L into C's first tile, its inverse into X).
void trailing_update_chol(int64_t n, const double* P, double* C, int64_t ld, double* X, int64_t ldx, int* info,
                          hipStream_t stream) {
  const unsigned tiles = static_cast<unsigned>((n + kT - 1) / kT);
  gemm64_kernel<double, double, true><<<dim3(tiles, tiles, 1), dim3(256), 0, stream>>>(
      n, n, int64_t{kT}, -1.0, P, ld, int64_t{1}, 0, P, int64_t{1}, ld, 0, 1.0, C, ld, int64_t{1}, 0, 1, X,
      ldx, info);
}

// Lower-triangular inverse X = L^-1 of a batch of n x n matrices (n a multiple
// of 64; batch stride s): the diagonal 64-blocks of X must already hold the
// inverses of L's, X's strictly upper part zero; tmp holds n^2 / 4 per batch.
// For a lower-triangular [L11 0; L21 L22] with X11 = L11^-1 and X22 = L22^-1,
// the missing block is X21 = -X22 (L21 X11).  A power-of-two size (64 2^j)
// joins its diagonal blocks pairwise up a binary tree, two b x b x b products
// per pair, batched over the pairs of a level (one matrix) or over the
// matrices (one launch per pair); any other size splits off its largest
// power-of-two leading block, inverts the rest recursively and joins the two.
void trtri_pow2(const double* L, double* X, int64_t n, int64_t ld, int64_t s, int batch, double* tmp,
                hipStream_t stream) {
  for (int64_t b = kT; b < n; b *= 2) {
    const int64_t pairs = n / (2 * b);
    const int64_t ps = 2 * b * (ld + 1);                  // diagonal step between pairs
    auto join = [&](int64_t off, int nbat, int64_t mstride) {
      gemm64(b, b, b, 1.0, L + off + b * ld, ld, int64_t{1}, X + off, ld, int64_t{1}, 0.0, tmp, b,
             int64_t{1}, stream, 0, nbat, mstride, mstride, b * b);
      gemm64(b, b, b, -1.0, X + off + b * ld + b, ld, int64_t{1}, tmp, b, int64_t{1}, 0.0, X + off + b * ld,
             ld, int64_t{1}, stream, 0, nbat, mstride, b * b, mstride);
    };
    if (batch == 1) {
      join(0, static_cast<int>(pairs), ps);
    } else {
      for (int64_t pr = 0; pr < pairs; ++pr) join(pr * ps, batch, s);
    }
  }
}

void trtri_lower(const double* L, double* X, int64_t n, int64_t ld, int64_t s, int batch, double* tmp,
                 hipStream_t stream) {
  int64_t n1 = kT;
  while (2 * n1 < n) n1 *= 2;
  if (2 * n1 == n || n1 == n) {
    trtri_pow2(L, X, n, ld, s, batch, tmp, stream);
    return;
  }
  const int64_t n2 = n - n1;                              // 0 < n2 < n1
  trtri_pow2(L, X, n1, ld, s, batch, tmp, stream);
  trtri_lower(L + n1 * (ld + 1), X + n1 * (ld + 1), n2, ld, s, batch, tmp, stream);
  gemm64(n2, n1, n1, 1.0, L + n1 * ld, ld, int64_t{1}, X, ld, int64_t{1}, 0.0, tmp, n1, int64_t{1}, stream, 0,
         batch, s, s, n2 * n1);
  gemm64(n2, n1, n2, -1.0, X + n1 * ld + n1, ld, int64_t{1}, tmp, n1, int64_t{1}, 0.0, X + n1 * ld, ld,
         int64_t{1}, stream, 0, batch, s, n2 * n1, s);
}

}  // namespace

// ---------------------------------------------------------------------------

sdq_status launch_hessian_accumulate(const float* x, int64_t m, int64_t k, double* h, hipStream_t stream) {
  // H[i][j] += 2 sum_p X[p][i] X[p][j]
  gemm64(k, k, m, 2.0, x, int64_t{1}, k, x, k, int64_t{1}, 1.0, h, k, int64_t{1}, stream, 2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "hessian launch");
  return SDQ_OK;
}

size_t hessian_factor_ws_bytes(int64_t k) {
  return 256 + align_up(static_cast<size_t>(k) * k * 8, 256) * 2 + align_up(static_cast<size_t>(k) * k * 2, 256);
}

sdq_status launch_hessian_factor(const double* h, int64_t k, double lam, double* u, void* ws,
                                 hipStream_t stream) {
  char* p = static_cast<char*>(ws);
  int* info = reinterpret_cast<int*>(p);
  double* A = reinterpret_cast<double*>(p + 256);
  double* X = reinterpret_cast<double*>(p + 256 + align_up(static_cast<size_t>(k) * k * 8, 256));
  double* tmp = reinterpret_cast<double*>(p + 256 + 2 * align_up(static_cast<size_t>(k) * k * 8, 256));
  const int64_t kk = k * k;
  clear_info_kernel<<<1, 64, 0, stream>>>(info);
  fill_f64_kernel<<<grid1(kk), 256, 0, stream>>>(X, kk, 0.0);
  reverse_tri_kernel<<<dim3(grid1(kk), 1), 256, 0, stream>>>(h, k, 0, k, A, k, 0, 1, lam);
  // Right-looking blocked Cholesky in 64-column steps: the panel below the
  // diagonal block is solved with the block's inverse, then the trailing lower
  // part is updated, and the same launch factors the next diagonal block.
  const int64_t t = k / kT;
  chol64_kernel<<<1, 256, 0, stream>>>(A, k, X, k, info);
  for (int64_t j = 0; j + 1 < t; ++j) {
    const int64_t d = j * kT, r0 = d + kT, rows = k - r0;
    // L[r0:, d] = A[r0:, d] L_dd^-T, in place
    gemm64(rows, int64_t{kT}, int64_t{kT}, 1.0, A + r0 * k + d, k, int64_t{1}, X + d * k + d, int64_t{1}, k,
           0.0, A + r0 * k + d, k, int64_t{1}, stream);
    // A[r0:, r0:] -= L[r0:, d] L[r0:, d]^T (lower), then block r0 factored
    trailing_update_chol(rows, A + r0 * k + d, A + r0 * k + r0, k, X + r0 * k + r0, k, info, stream);
  }
  trtri_lower(A, X, k, k, 0, 1, tmp, stream);
  reverse_tri_kernel<<<dim3(grid1(kk), 1), 256, 0, stream>>>(X, k, 0, k, u, k, 0, 0, 0.0);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "hessian factor launch");
  return SDQ_OK;
}

// Workspace of the compensated encoder: the plain encoder's, then (256-byte
// aligned) scratch row maxima, W64 (n x k), the fp32 block (n x B), E and G
// (n x B each), the scaled codes (n x M), and per block the reversed diagonal
// block of U, its inverse, the inverse reversed back (nb x B x B each) and
// the triangular-inverse scratch (nb x 64 x B).
struct CompWs {
  QuantWs q;
  uint32_t* rmax_scratch;
  double* w64;
  float* wblk;
  double* ebuf;
  double* gbuf;
  double* cb;
  double* lb;
  double* xb;
  double* vb;
  double* tmp;
};

size_t comp_ws_layout(const sdq_layout* L, CompWs* out, void* base) {
  char* p = static_cast<char*>(base);
  size_t off = align_up(quant_ws_layout(L, nullptr, nullptr), 256);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return p ? p + at : nullptr;
  };
  CompWs w;
  if (p) quant_ws_layout(L, &w.q, base);
  const size_t n = static_cast<size_t>(L->n), B = static_cast<size_t>(L->block), nb = static_cast<size_t>(L->nb);
  w.rmax_scratch = reinterpret_cast<uint32_t*>(take(static_cast<size_t>(L->n_pad) * 4));
  w.w64 = reinterpret_cast<double*>(take(n * L->k * 8));
  w.wblk = reinterpret_cast<float*>(take(n * B * 4));
  w.ebuf = reinterpret_cast<double*>(take(n * B * 8));
  w.gbuf = reinterpret_cast<double*>(take(n * B * 8));
  w.cb = reinterpret_cast<double*>(take(n * L->m_up * 8));
  w.lb = reinterpret_cast<double*>(take(nb * B * B * 8));
  w.xb = reinterpret_cast<double*>(take(nb * B * B * 8));
  w.vb = reinterpret_cast<double*>(take(nb * B * B * 8));
  w.tmp = reinterpret_cast<double*>(take(nb * kT * B * 8));
  if (out) *out = w;
  return off;
}

sdq_status launch_quantize_compensated(const float* w, const sdq_layout* L, const Tables* T,
                                       const double* u, int update, void* codes, float* scales, void* ws,
                                       hipStream_t stream) {
  CompWs cw;
  comp_ws_layout(L, &cw, ws);
  const int64_t n = L->n, k = L->k, B = L->block, nb = L->nb, M = L->m_up;
  // Base-3 layouts: every pass works on 2-bit fields in the workspace, which
  // are repacked at the end.
  const bool base3 = L->packing == SDQ_PACK_BASE3;
  const sdq_layout Fv = fields_view(L);
  const sdq_layout* F = &Fv;
  void* fcodes = base3 ? static_cast<void*>(cw.q.codes2) : codes;
  // 1. The plain encoding: row scales of the raw W, and block 0's final codes.
  clear_rmax(cw.q, L, stream);
  sdq_status st = launch_encode_blocks(w, k, 0, nb, F, T, fcodes, scales, cw.q, cw.q.rmax, cw.q.rmax, stream);
  if (st != SDQ_OK) return st;
  // 2. Joint update only: V_b = U_bb^-1 for every block: U_bb reversed is
  //    lower triangular; invert it (64-blocks, then the off-diagonal blocks)
  //    and reverse back.
  const int64_t bb = B * B;
  const bool joint = update == SDQ_COMP_JOINT;
  if (joint) {
    fill_f64_kernel<<<grid1(nb * bb), 256, 0, stream>>>(cw.xb, nb * bb, 0.0);
    reverse_tri_kernel<<<dim3(grid1(bb), static_cast<unsigned>(nb)), 256, 0, stream>>>(
        u, k, B * k + B, B, cw.lb, B, bb, 1, 0.0);
    trinv64_kernel<<<dim3(static_cast<unsigned>(B / kT), static_cast<unsigned>(nb)), 256, 0, stream>>>(
        cw.lb, B, kT * B + kT, bb, cw.xb, B, kT * B + kT, bb);
    trtri_lower(cw.lb, cw.xb, B, B, bb, static_cast<int>(nb), cw.tmp, stream);
    reverse_tri_kernel<<<dim3(grid1(bb), static_cast<unsigned>(nb)), 256, 0, stream>>>(
        cw.xb, B, bb, B, cw.vb, B, bb, 0, 0.0);
  }
  // 3. The walk over the blocks, W in fp64.
  widen_kernel<<<grid1(n * k), 256, 0, stream>>>(w, n * k, cw.w64);
  for (int64_t b = 0; b < nb; ++b) {
    extract_block_kernel<<<grid1(n * B), 256, 0, stream>>>(cw.w64, n, k, static_cast<int>(B), b * B,
                                                           cw.wblk, cw.ebuf);
    if (b > 0) {
      st = launch_encode_blocks(cw.wblk, B, b, 1, F, T, fcodes, scales, cw.q, cw.rmax_scratch,
                                cw.q.rmax, stream);
      if (st != SDQ_OK) return st;
    }
    if (b == nb - 1) break;
    unpack_scaled_kernel<<<grid1(n * M), 256, 0, stream>>>(static_cast<const uint32_t*>(fcodes), scales, n,
                                                           F->n_chunks, F->codes_per_chunk, F->bits,
                                                           b * M, static_cast<int>(M), cw.cb);
    // E_b = W_b - (s C_b) E^T
    gemm64(n, B, M, -1.0, cw.cb, M, int64_t{1}, T->e64, int64_t{1}, M, 1.0, cw.ebuf, B, int64_t{1}, stream);
    if (joint) {      // G = E_b V_b
      gemm64(n, B, B, 1.0, cw.ebuf, B, int64_t{1}, cw.vb + b * bb, B, int64_t{1}, 0.0, cw.gbuf, B, int64_t{1},
             stream);
    } else {          // G = E_b diag(U_bb)^-1
      divide_by_pivots_kernel<<<grid1(n * B), 256, 0, stream>>>(cw.ebuf, u, k, b * B, n, static_cast<int>(B),
                                                               cw.gbuf);
    }
    // W_F -= G U[Q, F]
    const int64_t f0 = (b + 1) * B;
    gemm64(n, k - f0, B, -1.0, cw.gbuf, B, int64_t{1}, u + b * B * k + f0, k, int64_t{1}, 1.0, cw.w64 + f0, k,
           int64_t{1}, stream);
  }
  if (base3) {
    st = launch_repack_base3(cw.q.codes2, L, codes, stream);
    if (st != SDQ_OK) return st;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "compensated encoder launch");
  return SDQ_OK;
}

size_t comp_ws_bytes(const sdq_layout* L) { return comp_ws_layout(L, nullptr, nullptr); }

}  // namespace sdq
