// libmgn kernels for CDNA4 (gfx950): one training step (forward and backward)
// of the MeshGraphNets encode-process-decode network on one partition.
//
// Kernel map (paper: section "Model", Algorithm 1; the paper's own code is
// PyTorch layers, these are fused replacements):
//   pack_kernel        parameter re-layout into MFMA fragment order
//   erecv / plan       per-edge receiver ids; receiver-aligned edge work units
//   rows_fwd           EncNode, EncEdge, node half of a block, DecNode
//   edge_fwd           edge half of a block: gather [e | v_s | v_r] into LDS,
//                      MLP on MFMA, LayerNorm, residual, ordered receiver sum
//   rows_bwd/edge_bwd  the same with the forward recomputed in-tile; the edge
//                      half ends at the first Linear's output gradient dz_0
//                      (edge-stream part applied, receiver sums formed)
//   input_grad         node gradients through that Linear's sender/receiver
//                      blocks: ordered per-node sums of dz_0 (transposed CSR
//                      for senders), then one node-level product
//   dw / dw_reduce     weight gradients as split-K MFMA GEMMs, fixed order
//   vec_reduce         bias and LayerNorm gradients, fixed order
//   mse                masked mean-squared-error loss and its gradient
// No float atomics anywhere: every sum has a fixed order, so results are
// bitwise reproducible run to run.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "../../include/mgn.h"

namespace mgn {

constexpr int NT = 256;          // threads per workgroup
constexpr int NW = NT / 64;      // waves per workgroup
constexpr int LDS_MAX = 160 * 1024;

template <int P>
struct PrecOf;
template <>
struct PrecOf<F32> {
  using type = PF32;
};
template <>
struct PrecOf<BF16> {
  using type = PBF16;
};

__host__ __device__ constexpr int rup(int x, int m) { return (x + m - 1) / m * m; }

// ------------------------------------------------------------ staging ---
// Loads 4 consecutive fp32 values and stores them to LDS in storage type.
template <class P>
__device__ __forceinline__ void st4(typename P::T* dst, float4 v) {
  if constexpr (sizeof(typename P::T) == 4) {
    *reinterpret_cast<float4*>(dst) = v;
  } else {
    uint2 w;
    w.x = (uint32_t)P::cvt(v.x) | ((uint32_t)P::cvt(v.y) << 16);
    w.y = (uint32_t)P::cvt(v.z) | ((uint32_t)P::cvt(v.w) << 16);
    *reinterpret_cast<uint2*>(dst) = w;
  }
}

// Copies `width` storage-type elements (a multiple of 16 bytes) from global
// row src into LDS row dst, one 16-byte chunk per thread of the group.
template <class P>
__device__ __forceinline__ void copy_row16(typename P::T* dst, const typename P::T* src, int width, int lane,
                                           int nlanes) {
  constexpr int E16 = 16 / sizeof(typename P::T);
  for (int c = lane * E16; c < width; c += nlanes * E16)
    *reinterpret_cast<uint4*>(dst + c) = *reinterpret_cast<const uint4*>(src + c);
}

// Copies n rows of `width` elements (16-byte multiple) from LDS (row stride
// ld) to consecutive global rows starting at dst, 16 bytes per thread.
template <class T, int NTH = NT>
__device__ __forceinline__ void store_rows(T* __restrict__ dst, const T* src, int ld, int n, int width) {
  constexpr int E16 = 16 / sizeof(T);
  const int cpr = width / E16;
  for (int i = threadIdx.x; i < n * cpr; i += NTH) {
    const int r = i / cpr, c = (i % cpr) * E16;
    *reinterpret_cast<uint4*>(dst + (int64_t)r * width + c) = *reinterpret_cast<const uint4*>(src + r * ld + c);
  }
}

// Stores an accumulator tile (MB x NBW blocks of 16x16) plus bias and
// optional ReLU into an LDS matrix of type OutT (row stride ld).
template <class P, int MB, int NBW, bool RELU, class OutT>
__device__ __forceinline__ void store_acc(const floatx4 (&acc)[MB][NBW], int nb0, const float* __restrict__ bias,
                                          int nvalid, OutT* dst, int ld) {
#pragma unroll
  for (int n = 0; n < NBW; ++n) {
    const int col = (nb0 + n) * 16 + acc_col();
    const float bv = (bias && col < nvalid) ? bias[col] : 0.f;
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = acc[m][n][r] + bv;
        if (RELU) v = v > 0.f ? v : 0.f;
        const int row = m * 16 + acc_row(r);
        if constexpr (__is_same(OutT, float)) {
          dst[row * ld + col] = v;
        } else {
          dst[row * ld + col] = P::cvt(v);
        }
      }
  }
}

// LayerNorm statistics of TM rows of width L (fp32 in LDS, row stride ld):
// replaces y by xhat = (y - mean) * rstd and stores rstd per row.  TPR
// consecutive threads share a row.
template <int TM, int L>
__device__ __forceinline__ void ln_normalise(float* Y, int ld, float eps, float* rstd_out) {
  constexpr int TPR = NT / TM;
  const int row = threadIdx.x / TPR, q = threadIdx.x % TPR;
  float* y = Y + row * ld;
  float s = 0.f;
  for (int c = q; c < L; c += TPR) s += y[c];
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o, 64);
  const float mu = s / L;
  float v = 0.f;
  for (int c = q; c < L; c += TPR) {
    const float d = y[c] - mu;
    v += d * d;
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) v += __shfl_xor(v, o, 64);
  const float rs = 1.0f / sqrtf(v / L + eps);
  for (int c = q; c < L; c += TPR) y[c] = (y[c] - mu) * rs;
  if (q == 0 && rstd_out) rstd_out[row] = rs;
}

// LayerNorm of TM rows in place: y <- gamma * (y - mean) * rstd + beta.
template <int TM, int L>
__device__ __forceinline__ void ln_rows(float* Y, int ld, float eps, const float* __restrict__ gamma,
                                        const float* __restrict__ beta) {
  constexpr int TPR = NT / TM;
  constexpr int PER = L / TPR;
  const int row = threadIdx.x / TPR, q = threadIdx.x % TPR;
  float* y = Y + row * ld;
  float v[PER];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    v[j] = y[q + j * TPR];
    s += v[j];
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o, 64);
  const float mu = s / L;
  float var = 0.f;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const float d = v[j] - mu;
    var += d * d;
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) var += __shfl_xor(var, o, 64);
  const float rs = 1.0f / sqrtf(var / L + eps);
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = q + j * TPR;
    y[c] = gamma[c] * ((v[j] - mu) * rs) + beta[c];
  }
}

template <int TM, int L>
__device__ __forceinline__ void ln_affine(float* Y, int ld, const float* __restrict__ gamma,
                                          const float* __restrict__ beta) {
  constexpr int TPR = NT / TM;
  const int row = threadIdx.x / TPR, q = threadIdx.x % TPR;
  float* y = Y + row * ld;
  for (int c = q; c < L; c += TPR) y[c] = gamma[c] * y[c] + beta[c];
}

// LayerNorm backward for TM rows: DM holds dL/d(LN output); XH holds xhat.
// Overwrites DM with dL/dy (y = LN input) and writes it in storage type to DY.
template <class P, int TM, int L>
__device__ __forceinline__ void ln_backward(float* DM, int ldm, const float* XH, int ldx, const float* rstd,
                                            const float* __restrict__ gamma, typename P::T* DY, int ldy) {
  constexpr int TPR = NT / TM;
  const int row = threadIdx.x / TPR, q = threadIdx.x % TPR;
  float* dm = DM + row * ldm;
  const float* xh = XH + row * ldx;
  float s1 = 0.f, s2 = 0.f;
  for (int c = q; c < L; c += TPR) {
    const float d = dm[c] * gamma[c];
    s1 += d;
    s2 += d * xh[c];
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) {
    s1 += __shfl_xor(s1, o, 64);
    s2 += __shfl_xor(s2, o, 64);
  }
  const float m1 = s1 / L, m2 = s2 / L, rs = rstd[row];
  for (int c = q; c < L; c += TPR) {
    const float dy = rs * (dm[c] * gamma[c] - m1 - xh[c] * m2);
    dm[c] = dy;
    DY[row * ldy + c] = P::cvt(dy);
  }
}

// Column sums over TM rows with a fixed (ascending) row order.
__device__ __forceinline__ float col_sum(const float* A, int ld, int rows, int c) {
  float s = 0.f;
  for (int r = 0; r < rows; ++r) s += A[r * ld + c];
  return s;
}

// Sum of acc over the tile's rows for each of the wave's columns (all lanes
// of a 16-lane column group end with the same value).
template <int MB, int NBW>
__device__ __forceinline__ void acc_colsum(const floatx4 (&acc)[MB][NBW], float (&out)[NBW]) {
#pragma unroll
  for (int n = 0; n < NBW; ++n) {
    float s = 0.f;
#pragma unroll
    for (int m = 0; m < MB; ++m) s += (acc[m][n][0] + acc[m][n][1]) + (acc[m][n][2] + acc[m][n][3]);
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    out[n] = s;
  }
}

// Row totals over all L columns of a wave-column-split tile (MB row blocks of
// 16; wave w holds the 16-column blocks w*NBW ..).  v[q][m][r] enters as this
// lane's partial of row m*16 + acc_row(r) and leaves as the row's total, with
// the same bits in every lane that holds the row: the 16 lanes of a row group
// combine by a butterfly (commutative pairs), the waves through LDS slots
// red[NW][Q][MB*16] in ascending wave order.
template <int Q, int MB, int NWAVES = NW>
__device__ __forceinline__ void row_totals(float (&v)[Q][MB][4], float* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = v[q][m][r];
        x += __shfl_xor(x, 1, 64);
        x += __shfl_xor(x, 2, 64);
        x += __shfl_xor(x, 4, 64);
        x += __shfl_xor(x, 8, 64);
        v[q][m][r] = x;
      }
  if ((lane & 15) == 0) {
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[((wave * Q + q) * MB + m) * 16 + acc_row(r)] = v[q][m][r];
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = 0.f;
#pragma unroll
        for (int w = 0; w < NWAVES; ++w) x += red[((w * Q + q) * MB + m) * 16 + acc_row(r)];
        v[q][m][r] = x;
      }
}

// LayerNorm statistics on an accumulator tile (bias already added): y
// becomes xhat = (y - mean) * rstd, with the two-pass variance; rstd of the
// lane's rows is returned.  Uses two disjoint slot sets red0, red1.
template <int MB, int NBW, int L, int NWAVES = NW>
__device__ __forceinline__ void ln_tile(floatx4 (&y)[MB][NBW], float eps, float* red0, float* red1,
                                        float (&rs)[MB][4]) {
  float s[1][MB][4], v[1][MB][4];
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float x = 0.f;
#pragma unroll
      for (int n = 0; n < NBW; ++n) x += y[m][n][r];
      s[0][m][r] = x;
    }
  row_totals<1, MB, NWAVES>(s, red0);
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float mu = s[0][m][r] / L;
      float x = 0.f;
#pragma unroll
      for (int n = 0; n < NBW; ++n) {
        const float d = y[m][n][r] - mu;
        x += d * d;
      }
      s[0][m][r] = mu;
      v[0][m][r] = x;
    }
  row_totals<1, MB, NWAVES>(v, red1);
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      rs[m][r] = 1.0f / sqrtf(v[0][m][r] / L + eps);
#pragma unroll
      for (int n = 0; n < NBW; ++n) y[m][n][r] = (y[m][n][r] - s[0][m][r]) * rs[m][r];
    }
}

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(uint16_t x) { return bf2f(x); }

// ----------------------------------------------------------------- pack ---
template <class P>
__global__ void pack_kernel(const float* __restrict__ W, int out, int in, int bwd, uint4* __restrict__ dst,
                            int nkg, int64_t total) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  const int kg = (int)((idx >> 6) % nkg);
  const int nb = (int)((idx >> 6) / nkg);
  const int j = nb * 16 + (lane & 15);
  const int k0 = kg * P::KG + (lane >> 4) * P::EL;
  typename P::T v[P::EL];
#pragma unroll
  for (int e = 0; e < P::EL; ++e) {
    const int k = k0 + e;
    float x = 0.f;
    if (!bwd) {
      if (j < out && k < in) x = W[(int64_t)j * in + k];
    } else {
      if (j < in && k < out) x = W[(int64_t)k * in + j];
    }
    v[e] = P::cvt(x);
  }
  dst[idx] = *reinterpret_cast<const uint4*>(v);
}

// ------------------------------------------------------------- fills ---
// Plain fill kernels (used instead of memset nodes, which some callers
// capture into graphs).
__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}
__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

hipError_t launch_zero(float* p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t g = (n + NT - 1) / NT;
  hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)(g < 4096 ? g : 4096)), dim3(NT), 0, st, p, n, 0.f);
  return hipGetLastError();
}

// bf16 copy of the halo latents of every block: V16[k][n_owned + h] = H[k][h].
__global__ void halo_bf16_kernel(const float* __restrict__ H, int K, int64_t n_halo, int64_t n_owned, int L,
                                 uint16_t* __restrict__ V16, int64_t stride) {
  const int64_t per = n_halo * L / 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < (int64_t)K * per;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = i / per, j = i % per;
    const float4 v = reinterpret_cast<const float4*>(H + k * n_halo * L)[j];
    uint2 w;
    w.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
    w.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
    reinterpret_cast<uint2*>(V16 + k * stride + n_owned * L)[j] = w;
  }
}

hipError_t launch_halo_bf16(const float* H, int K, int64_t n_halo, int64_t n_owned, int L, void* V16,
                            int64_t v16_block_stride, hipStream_t st) {
  const int64_t n = (int64_t)K * n_halo * L / 4;
  if (n == 0) return hipSuccess;
  const int64_t g = (n + NT - 1) / NT;
  hipLaunchKernelGGL(halo_bf16_kernel, dim3((unsigned)(g < 8192 ? g : 8192)), dim3(NT), 0, st, H, K, n_halo, n_owned,
                     L, reinterpret_cast<uint16_t*>(V16), v16_block_stride);
  return hipGetLastError();
}

// ------------------------------------------------------------ update ---
// Algorithm 1's parameter update: p <- p - lr * g, one fused multiply-add
// (one rounding) per entry.
__global__ void sgd_kernel(float* __restrict__ p, const float* __restrict__ g, int64_t n, float lr) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = __builtin_fmaf(-lr, g[i], p[i]);
}

hipError_t launch_sgd(float* p, const float* g, int64_t n, float lr, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t b = (n + NT - 1) / NT;
  hipLaunchKernelGGL(sgd_kernel, dim3((unsigned)(b < 4096 ? b : 4096)), dim3(NT), 0, st, p, g, n, lr);
  return hipGetLastError();
}

// Next-step rollout: the flow columns of the node features take the
// predicted increment, nf[i][col0 + j] += out[i][j].
__global__ void rollout_kernel(const float* __restrict__ out, int64_t n, int d, float* __restrict__ nf, int fin,
                               int col0) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n * d; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / d;
    const int j = (int)(t - i * d);
    nf[i * fin + col0 + j] += out[t];
  }
}

hipError_t launch_rollout(const float* out, int64_t n, int d, float* nf, int fin, int col0, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t b = (n * d + NT - 1) / NT;
  hipLaunchKernelGGL(rollout_kernel, dim3((unsigned)(b < 8192 ? b : 8192)), dim3(NT), 0, st, out, n, d, nf, fin, col0);
  return hipGetLastError();
}

// ------------------------------------------------------------ Normalize ---
// Online standardisation per feature column (Normalize of Algorithm 1):
// stats = [n, column sums, column sums of squares] in fp64.  Accumulation:
// up to NORM_BLOCKS workgroups, each over a contiguous row range; thread t
// takes column t % cols of every (NT / cols)-th row from its group's first
// (consecutive threads read consecutive floats), with fp64 sums; the groups'
// sums and then the workgroups' partials are added in a fixed order (no
// atomics), so the result does not depend on timing.
constexpr int NORM_BLOCKS = 512;

__global__ __launch_bounds__(NT) void norm_partial_kernel(const float* __restrict__ x, int64_t rows, int cols,
                                                          double* __restrict__ part) {
  __shared__ double s1[NT], s2[NT];
  const int G = NT / cols;  // row groups of the workgroup
  const int t = threadIdx.x, g = t / cols, c = t - g * cols;
  const int64_t r0 = rows * blockIdx.x / gridDim.x, r1 = rows * (blockIdx.x + 1) / gridDim.x;
  double a = 0.0, b = 0.0;
  if (g < G)
    for (int64_t r = r0 + g; r < r1; r += G) {
      const double v = x[r * cols + c];
      a += v;
      b += v * v;
    }
  s1[t] = a;
  s2[t] = b;
  __syncthreads();
  if (t < cols) {
    double A = 0.0, B = 0.0;
    for (int k = 0; k < G; ++k) {
      A += s1[k * cols + t];
      B += s2[k * cols + t];
    }
    part[(int64_t)blockIdx.x * 2 * cols + t] = A;
    part[(int64_t)blockIdx.x * 2 * cols + cols + t] = B;
  }
}

// stats[1 + j] += sum over the workgroups, in order, of part[b][j] (j < 2 cols:
// the column sums, then the sums of squares); stats[0] += rows.
__global__ void norm_final_kernel(const double* __restrict__ part, int nb, int cols, int64_t rows,
                                  double* __restrict__ stats) {
  const int t = threadIdx.x;
  if (t < 2 * cols) {
    double A = 0.0;
    for (int b = 0; b < nb; ++b) A += part[(int64_t)b * 2 * cols + t];
    stats[1 + t] += A;
  }
  if (t == 0) stats[0] += (double)rows;
}

// out = (x - mean) / max(std, eps) per column, in fp64, rounded once; out may be x.
__global__ void norm_apply_kernel(const float* x, int64_t n, int cols, const double* __restrict__ stats, double eps,
                                  float* out) {
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / cols;
    const int c = (int)(t - i * cols);
    double mean = 0.0, sd = 1.0;
    if (stats[0] > 0) {
      mean = stats[1 + c] / stats[0];
      const double var = stats[1 + cols + c] / stats[0] - mean * mean;
      sd = sqrt(var > 0 ? var : 0.0);
      if (sd < eps) sd = eps;
    }
    out[t] = (float)((x[t] - mean) / sd);
  }
}

int norm_work_doubles(int cols) { return NORM_BLOCKS * 2 * cols; }
static_assert(NORM_BLOCKS * 2 == MGN_NORM_WORK_PER_COL && MGN_NORM_MAX_COLS * 2 <= NT, "Normalize sizes");

hipError_t launch_norm_accumulate(const float* x, int64_t rows, int cols, double* stats, double* work,
                                  hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (cols < 1 || cols > NT) return hipErrorInvalidValue;
  const int64_t want = (rows + 1023) / 1024;
  const int nb = (int)(want < NORM_BLOCKS ? want : NORM_BLOCKS);
  hipLaunchKernelGGL(norm_partial_kernel, dim3(nb), dim3(NT), 0, st, x, rows, cols, work);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(norm_final_kernel, dim3(1), dim3(NT), 0, st, work, nb, cols, rows, stats);
  return hipGetLastError();
}

hipError_t launch_norm_apply(const float* x, int64_t rows, int cols, const double* stats, double eps, float* out,
                             hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int64_t n = rows * cols, b = (n + NT - 1) / NT;
  hipLaunchKernelGGL(norm_apply_kernel, dim3((unsigned)(b < 8192 ? b : 8192)), dim3(NT), 0, st, x, n, cols, stats,
                     eps, out);
  return hipGetLastError();
}

// ------------------------------------------------------- halo exchange ---
// Row copy between two node-row buffers of width L = 4 * L4 floats, the
// one-GPU form of Algorithm 1's pack / exchange / unpack:
// dst[dst_rows[i]] = src[src_rows[i]] (add == 0) or += (add == 1).  A pair
// with an index outside [0, n_src) or [0, n_dst) is skipped.
__global__ void rows_copy_kernel(const float* __restrict__ src, int64_t n_src, const int32_t* __restrict__ src_rows,
                                 const int32_t* __restrict__ dst_rows, int64_t n, int L4, float* __restrict__ dst,
                                 int64_t n_dst, int add) {
  const int64_t total = n * L4;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / L4;
    const int c = (int)(t - i * L4);
    const int32_t s = src_rows[i], d = dst_rows[i];
    if (s < 0 || s >= n_src || d < 0 || d >= n_dst) continue;
    const float4 v = reinterpret_cast<const float4*>(src + (int64_t)s * L4 * 4)[c];
    float4* q = reinterpret_cast<float4*>(dst + (int64_t)d * L4 * 4) + c;
    if (add) {
      float4 o = *q;
      o.x += v.x;
      o.y += v.y;
      o.z += v.z;
      o.w += v.w;
      *q = o;
    } else {
      *q = v;
    }
  }
}

hipError_t launch_rows_copy(const float* src, int64_t n_src, const int32_t* src_rows, const int32_t* dst_rows,
                            int64_t n, int L, float* dst, int64_t n_dst, int add, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t g = (n * (L / 4) + NT - 1) / NT;
  hipLaunchKernelGGL(rows_copy_kernel, dim3((unsigned)(g < 8192 ? g : 8192)), dim3(NT), 0, st, src, n_src, src_rows,
                     dst_rows, n, L / 4, dst, n_dst, add);
  return hipGetLastError();
}

// ------------------------------------------------------------- planning ---
__global__ void erecv_kernel(const int32_t* __restrict__ row_ptr, int64_t n_owned, int32_t* __restrict__ erecv) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n_owned) return;
  for (int32_t e = row_ptr[r]; e < row_ptr[r + 1]; ++e) erecv[e] = (int32_t)r;
}

constexpr int PLAN_CHUNK = 128;  // receivers per planning thread

// Greedy packing of consecutive receivers into work units of at most
// te_target edges and r_max receivers (a receiver with more edges than
// te_target gets a unit of its own); chunk boundaries close a unit.
__device__ int plan_chunk(const int32_t* row_ptr, int64_t r0, int64_t r1, int te_target, int r_max,
                          int32_t* out) {
  int count = 0, edges = 0, recv = 0;
  for (int64_t r = r0; r < r1; ++r) {
    const int d = row_ptr[r + 1] - row_ptr[r];
    if (recv > 0 && (edges + d > te_target || recv + 1 > r_max)) {
      edges = 0;
      recv = 0;
    }
    if (recv == 0) {
      if (out) out[count] = (int32_t)r;
      ++count;
    }
    edges += d;
    recv += 1;
  }
  return count;
}

__global__ void plan_count_kernel(const int32_t* __restrict__ row_ptr, int64_t n_owned, int te_target, int r_max,
                                  int32_t* __restrict__ cnt, int64_t nch) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nch) return;
  const int64_t r0 = c * PLAN_CHUNK, r1 = r0 + PLAN_CHUNK < n_owned ? r0 + PLAN_CHUNK : n_owned;
  cnt[c] = plan_chunk(row_ptr, r0, r1, te_target, r_max, nullptr);
}

// Exclusive scan of the chunk counts in one workgroup (fixed order).
__global__ void plan_scan_kernel(int32_t* __restrict__ cnt, int64_t nch, int32_t* __restrict__ n_units) {
  __shared__ int32_t part[NT];
  const int t = threadIdx.x;
  const int64_t per = (nch + NT - 1) / NT;
  const int64_t b = t * per, e = b + per < nch ? b + per : nch;
  int32_t s = 0;
  for (int64_t i = b; i < e; ++i) s += cnt[i];
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int32_t acc = 0;
    for (int i = 0; i < NT; ++i) {
      const int32_t v = part[i];
      part[i] = acc;
      acc += v;
    }
    *n_units = acc;
  }
  __syncthreads();
  int32_t acc = part[t];
  for (int64_t i = b; i < e; ++i) {
    const int32_t v = cnt[i];
    cnt[i] = acc;
    acc += v;
  }
}

__global__ void plan_write_kernel(const int32_t* __restrict__ row_ptr, int64_t n_owned, int te_target, int r_max,
                                  const int32_t* __restrict__ off, int64_t nch, const int32_t* __restrict__ n_units,
                                  int32_t* __restrict__ unit_r) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= nch) return;
  const int64_t r0 = c * PLAN_CHUNK, r1 = r0 + PLAN_CHUNK < n_owned ? r0 + PLAN_CHUNK : n_owned;
  plan_chunk(row_ptr, r0, r1, te_target, r_max, unit_r + off[c]);
  if (c == nch - 1) unit_r[*n_units] = (int32_t)n_owned;
}

// ---------------------------------------------------------- row kernels ---
template <int KIND, int L>
struct RowShape {
  static constexpr int KIN = (KIND == ENC_NODE || KIND == ENC_EDGE) ? 32 : (KIND == NODE_BLOCK ? 2 * L : L);
  static constexpr int NOUT = (KIND == DECODER) ? 16 : L;
  static constexpr bool LN = KIND != DECODER;
};

// LDS layout of a row kernel with TM rows (bytes).  X: inputs; HB, HC: hidden
// activations; Y: last-layer output / xhat (aliased onto X when it fits);
// DY: gradient in storage type; DM: fp32 gradient / output staging.
template <class P, int KIND, int L, int D, int TM>
struct RowLds {
  using S = RowShape<KIND, L>;
  static constexpr int LDX = S::KIN + P::PAD;
  static constexpr int LDH = L + P::PAD;
  static constexpr int LDY = S::NOUT + 4;
  static constexpr int LDM = (S::NOUT > L ? S::NOUT : L) + 4;
  static constexpr int XB = TM * LDX * (int)sizeof(typename P::T);
  static constexpr int HB = TM * LDH * (int)sizeof(typename P::T);
  static constexpr int YB = TM * LDY * 4;
  static constexpr int MB = TM * LDM * 4;
  static constexpr bool Y_IN_X = XB >= YB;
  static constexpr int OFF_H = rup(XB, 16);
  static constexpr int OFF_H2 = OFF_H + HB;
  static constexpr int OFF_Y = Y_IN_X ? 0 : OFF_H2 + (D == 3 ? HB : 0);
  static constexpr int END_F = Y_IN_X ? OFF_H2 + (D == 3 ? HB : 0) : OFF_Y + YB;  // forward kernels
  static constexpr int OFF_DY = rup(END_F, 16);
  static constexpr int OFF_DM = OFF_DY + HB;
  static constexpr int OFF_RS = OFF_DM + MB;
  static constexpr int END_B = OFF_RS + TM * 4;  // backward kernels
};

template <class P, int KIND, int L, int D>
struct RowTM {
  static constexpr int value = RowLds<P, KIND, L, D, 64>::END_B <= LDS_MAX   ? 64
                               : RowLds<P, KIND, L, D, 32>::END_B <= LDS_MAX ? 32
                                                                             : 16;
};

// Stages the first Linear's input rows into LDS X (zero rows past `n`).
template <class P, int KIND, int L, int TM, int LDX>
__device__ __forceinline__ void stage_rows(typename P::T* X, const float* __restrict__ in0,
                                           const float* __restrict__ in1, int fin, int64_t row0, int n,
                                           const uint16_t* __restrict__ in0_16 = nullptr) {
  using S = RowShape<KIND, L>;
  if constexpr (KIND == ENC_NODE || KIND == ENC_EDGE) {
    for (int i = threadIdx.x; i < TM * S::KIN; i += NT) {
      const int r = i / S::KIN, c = i % S::KIN;
      const float v = (r < n && c < fin) ? in0[(row0 + r) * fin + c] : 0.f;
      X[r * LDX + c] = P::cvt(v);
    }
  } else {
    constexpr int Q = L / 4;  // float4 per source row
    constexpr int NSRC = KIND == NODE_BLOCK ? 2 : 1;
    constexpr int IT = (TM * Q * NSRC + NT - 1) / NT;
    float4 v[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int i = threadIdx.x + j * NT, r = i / (Q * NSRC), rem = i % (Q * NSRC), s = rem / Q, c4 = rem % Q;
      v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (i < TM * Q * NSRC && r < n) {
        if (s == 0 && in0_16) {  // bf16 copy of the node rows (exact in the bf16 operand type)
          const uint2 w = reinterpret_cast<const uint2*>(in0_16 + (row0 + r) * L)[c4];
          v[j] = make_float4(bf2f((uint16_t)w.x), bf2f((uint16_t)(w.x >> 16)), bf2f((uint16_t)w.y),
                             bf2f((uint16_t)(w.y >> 16)));
        } else {
          v[j] = reinterpret_cast<const float4*>((s == 0 ? in0 : in1) + (row0 + r) * L)[c4];
        }
      }
    }
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int i = threadIdx.x + j * NT, r = i / (Q * NSRC), rem = i % (Q * NSRC), s = rem / Q, c4 = rem % Q;
      if (i < TM * Q * NSRC) st4<P>(X + r * LDX + s * L + c4 * 4, v[j]);
    }
  }
}

// Forward of the MLP on a staged tile: X -> ... -> Y (fp32, last layer + bias,
// before LayerNorm).  Hidden activations stay in HB (and HC for depth 3).
template <class P, int KIND, int L, int D, int TM>
__device__ __forceinline__ void mlp_tile_forward(const Mlp& mlp, typename P::T* X, typename P::T* HB,
                                                 typename P::T* HC, float* Y, int ldx, int ldh, int ldy) {
  using S = RowShape<KIND, L>;
  constexpr int MB = TM / 16;
  constexpr int NBW = L / 16 / NW > 0 ? L / 16 / NW : 1;
  const int wave = threadIdx.x >> 6;
  {
    floatx4 acc[MB][NBW];
    if (wave * NBW * 16 < L) {
      if constexpr (KIND == ENC_NODE || KIND == ENC_EDGE)
        wave_gemm<P, MB, NBW>(X, ldx, mlp.lin[0].wf, mlp.lin[0].nkgf, wave * NBW, acc);
      else
        wave_gemm_k<P, MB, NBW, S::KIN / P::KG>(X, ldx, mlp.lin[0].wf, wave * NBW, acc);
      store_acc<P, MB, NBW, true>(acc, wave * NBW, mlp.lin[0].b, L, HB, ldh);
    }
  }
  __syncthreads();
  typename P::T* hin = HB;
  if constexpr (D == 3) {
    floatx4 acc[MB][NBW];
    if (wave * NBW * 16 < L) {
      wave_gemm_k<P, MB, NBW, L / P::KG>(HB, ldh, mlp.lin[1].wf, wave * NBW, acc);
      store_acc<P, MB, NBW, true>(acc, wave * NBW, mlp.lin[1].b, L, HC, ldh);
    }
    __syncthreads();
    hin = HC;
  }
  {
    constexpr int NB_OUT = S::NOUT / 16;
    constexpr int NBO = NB_OUT / NW > 0 ? NB_OUT / NW : 1;
    floatx4 acc[MB][NBO];
    if (wave * NBO < NB_OUT) {
      wave_gemm_k<P, MB, NBO, L / P::KG>(hin, ldh, mlp.lin[D - 1].wf, wave * NBO, acc);
      store_acc<P, MB, NBO, false>(acc, wave * NBO, mlp.lin[D - 1].b, mlp.lin[D - 1].out, Y, ldy);
    }
  }
  __syncthreads();
}

template <int P_, int L, int D, int KIND>
__global__ __launch_bounds__(NT) void rows_fwd_kernel(RowsFwdArgs a) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  constexpr int TM = RowTM<P, KIND, L, D>::value;
  using Lay = RowLds<P, KIND, L, D, TM>;
  extern __shared__ __align__(16) unsigned char lds[];
  T* X = reinterpret_cast<T*>(lds);
  T* HB = reinterpret_cast<T*>(lds + Lay::OFF_H);
  T* HC = reinterpret_cast<T*>(lds + Lay::OFF_H2);
  float* Y = reinterpret_cast<float*>(lds + Lay::OFF_Y);
  const int64_t ntiles = (a.rows + TM - 1) / TM;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t row0 = tile * TM;
    const int n = (int)(a.rows - row0 < TM ? a.rows - row0 : TM);
    stage_rows<P, KIND, L, TM, Lay::LDX>(X, a.in0, a.in1, a.fin, row0, n);
    __syncthreads();
    mlp_tile_forward<P, KIND, L, D, TM>(a.mlp, X, HB, HC, Y, Lay::LDX, Lay::LDH, Lay::LDY);
    if constexpr (RowShape<KIND, L>::LN) {
      ln_rows<TM, L>(Y, Lay::LDY, a.eps, a.mlp.gamma, a.mlp.beta);
      __syncthreads();
    }
    if constexpr (KIND == DECODER) {
      float* out = reinterpret_cast<float*>(a.out);
      for (int i = threadIdx.x; i < n * a.fout; i += NT) {
        const int r = i / a.fout, c = i % a.fout;
        out[(row0 + r) * a.fout + c] = Y[r * Lay::LDY + c];
      }
    } else if constexpr (KIND == ENC_EDGE) {
      T* out = reinterpret_cast<T*>(a.out);
      for (int i = threadIdx.x; i < n * L; i += NT) {
        const int r = i / L, c = i % L;
        out[(row0 + r) * L + c] = P::cvt(Y[r * Lay::LDY + c]);
      }
    } else {
      float* out = reinterpret_cast<float*>(a.out);
      uint16_t* out16 = reinterpret_cast<uint16_t*>(a.out16);
      constexpr int Q = L / 4;
      for (int i = threadIdx.x; i < n * Q; i += NT) {
        const int r = i / Q, c4 = i % Q;
        float4 y = *reinterpret_cast<const float4*>(Y + r * Lay::LDY + c4 * 4);
        if constexpr (KIND == NODE_BLOCK) {
          const float4 v = reinterpret_cast<const float4*>(a.in0 + (row0 + r) * L)[c4];
          y.x += v.x;
          y.y += v.y;
          y.z += v.z;
          y.w += v.w;
        }
        reinterpret_cast<float4*>(out + (row0 + r) * L)[c4] = y;
        if (out16) {
          uint2 w;
          w.x = (uint32_t)f2bf(y.x) | ((uint32_t)f2bf(y.y) << 16);
          w.y = (uint32_t)f2bf(y.z) | ((uint32_t)f2bf(y.w) << 16);
          reinterpret_cast<uint2*>(out16 + (row0 + r) * L)[c4] = w;
        }
      }
    }
    __syncthreads();
  }
}

// Backward of a row MLP with the forward recomputed in-tile.
template <int P_, int L, int D, int KIND>
__global__ __launch_bounds__(NT) void rows_bwd_kernel(RowsBwdArgs a) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  using S = RowShape<KIND, L>;
  constexpr int TM = RowTM<P, KIND, L, D>::value;
  using Lay = RowLds<P, KIND, L, D, TM>;
  constexpr int MB = TM / 16;
  constexpr int NBW = L / 16 / NW > 0 ? L / 16 / NW : 1;
  extern __shared__ __align__(16) unsigned char lds[];
  T* X = reinterpret_cast<T*>(lds);
  T* HB = reinterpret_cast<T*>(lds + Lay::OFF_H);
  T* HC = reinterpret_cast<T*>(lds + Lay::OFF_H2);
  float* Y = reinterpret_cast<float*>(lds + Lay::OFF_Y);
  T* DY = reinterpret_cast<T*>(lds + Lay::OFF_DY);
  float* DM = reinterpret_cast<float*>(lds + Lay::OFF_DM);
  float* RS = reinterpret_cast<float*>(lds + Lay::OFF_RS);
  const int wave = threadIdx.x >> 6;
  const bool wave_has_cols = wave * NBW * 16 < L;
  const int tid = threadIdx.x;
  const int nout_last = a.mlp.lin[D - 1].out;

  // per-workgroup vector gradient accumulators
  float g_gamma = 0.f, g_beta = 0.f, g_blast = 0.f;  // column tid
  float g_bh[2][NBW];                                  // hidden-layer biases, columns of this wave
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int n = 0; n < NBW; ++n) g_bh[j][n] = 0.f;

  const int64_t ntiles = (a.rows + TM - 1) / TM;
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t row0 = tile * TM;
    const int n = (int)(a.rows - row0 < TM ? a.rows - row0 : TM);
    stage_rows<P, KIND, L, TM, Lay::LDX>(X, a.in0, a.in1, a.fin, row0, n,
                                         reinterpret_cast<const uint16_t*>(a.in0_16));
    // incoming gradient (zero rows past n; decoder: dOut padded to 16 columns)
    for (int i = tid; i < TM * S::NOUT; i += NT) {
      const int r = i / S::NOUT, c = i % S::NOUT;
      float v = 0.f;
      if (r < n) {
        if constexpr (KIND == DECODER) {
          if (c < a.fout) v = a.dm[(row0 + r) * a.fout + c];
        } else {
          v = a.dm16 ? bf2f(a.dm16[(row0 + r) * L + c]) : a.dm[(row0 + r) * L + c];
        }
      }
      DM[r * Lay::LDM + c] = v;
    }
    __syncthreads();
    if constexpr (S::LN) {
      mlp_tile_forward<P, KIND, L, D, TM>(a.mlp, X, HB, HC, Y, Lay::LDX, Lay::LDH, Lay::LDY);
      ln_normalise<TM, L>(Y, Lay::LDY, a.eps, RS);
      __syncthreads();
      if (tid < L) {
        for (int r = 0; r < n; ++r) {
          const float d = DM[r * Lay::LDM + tid];
          g_gamma += d * Y[r * Lay::LDY + tid];
          g_beta += d;
        }
      }
      __syncthreads();
      ln_backward<P, TM, L>(DM, Lay::LDM, Y, Lay::LDY, RS, a.mlp.gamma, DY, Lay::LDH);
      __syncthreads();
      if (tid < L) g_blast += col_sum(DM, Lay::LDM, n, tid);
    } else {
      // decoder: only the hidden activations are needed
      {
        floatx4 acc[MB][NBW];
        if (wave_has_cols) {
          wave_gemm_k<P, MB, NBW, S::KIN / P::KG>(X, Lay::LDX, a.mlp.lin[0].wf, wave * NBW, acc);
          store_acc<P, MB, NBW, true>(acc, wave * NBW, a.mlp.lin[0].b, L, HB, Lay::LDH);
        }
      }
      __syncthreads();
      if constexpr (D == 3) {
        floatx4 acc[MB][NBW];
        if (wave_has_cols) {
          wave_gemm_k<P, MB, NBW, L / P::KG>(HB, Lay::LDH, a.mlp.lin[1].wf, wave * NBW, acc);
          store_acc<P, MB, NBW, true>(acc, wave * NBW, a.mlp.lin[1].b, L, HC, Lay::LDH);
        }
        __syncthreads();
      }
      // gradient at the decoder output, zero past the 16 padded columns up to
      // one full k-group of the backward GEMM
      for (int i = tid; i < TM * 32; i += NT) {
        const int r = i / 32, c = i % 32;
        DY[r * Lay::LDH + c] = P::cvt(c < 16 ? DM[r * Lay::LDM + c] : 0.f);
      }
      if (tid < nout_last) g_blast += col_sum(DM, Lay::LDM, n, tid);
      __syncthreads();
    }
    // gradient at the last Linear's output and the hidden activations, for the
    // weight-gradient GEMMs
    store_rows(reinterpret_cast<T*>(a.delta[D - 1]) + row0 * S::NOUT, DY, Lay::LDH, n, S::NOUT);
    store_rows(reinterpret_cast<T*>(a.hid[0]) + row0 * L, HB, Lay::LDH, n, L);
    if constexpr (D == 3) store_rows(reinterpret_cast<T*>(a.hid[1]) + row0 * L, HC, Lay::LDH, n, L);
    // back through the hidden layers: dz_{j-1} = (dz_j W_j) * [h_{j-1} > 0]
#pragma unroll
    for (int j = D - 1; j >= 1; --j) {
      const T* hprev = (j == 2) ? HC : HB;
      floatx4 acc[MB][NBW];
      if (wave_has_cols) {
        if (KIND == DECODER && j == D - 1)
          wave_gemm_k<P, MB, NBW, 1>(DY, Lay::LDH, a.mlp.lin[j].wb, wave * NBW, acc);
        else
          wave_gemm_k<P, MB, NBW, L / P::KG>(DY, Lay::LDH, a.mlp.lin[j].wb, wave * NBW, acc);
      }
      __syncthreads();
      if (wave_has_cols) {
#pragma unroll
        for (int nn = 0; nn < NBW; ++nn)
#pragma unroll
          for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = m * 16 + acc_row(r), col = (wave * NBW + nn) * 16 + acc_col();
              const float h = P::tof(hprev[row * Lay::LDH + col]);
              acc[m][nn][r] = h > 0.f ? acc[m][nn][r] : 0.f;
              DY[row * Lay::LDH + col] = P::cvt(acc[m][nn][r]);
            }
        float cs[NBW];
        acc_colsum<MB, NBW>(acc, cs);
#pragma unroll
        for (int nn = 0; nn < NBW; ++nn) g_bh[j - 1][nn] += cs[nn];
      }
      __syncthreads();
      store_rows(reinterpret_cast<T*>(a.delta[j - 1]) + row0 * L, DY, Lay::LDH, n, L);
    }
    // input gradients
    if constexpr (KIND == NODE_BLOCK || KIND == DECODER) {
      constexpr int NPASS = KIND == NODE_BLOCK ? 2 : 1;
#pragma unroll
      for (int pass = 0; pass < NPASS; ++pass) {
        floatx4 acc[MB][NBW];
        if (wave_has_cols)
          wave_gemm_k<P, MB, NBW, L / P::KG>(DY, Lay::LDH, a.mlp.lin[0].wb, pass * (L / 16) + wave * NBW, acc);
        __syncthreads();  // DM (gradient staging) may still be read above
        if (wave_has_cols) store_acc<P, MB, NBW, false>(acc, wave * NBW, nullptr, L, DM, Lay::LDM);
        __syncthreads();
        float* dst = pass == 0 ? a.dx0 : a.dx1;
        constexpr int Q = L / 4;
        for (int i = tid; i < n * Q; i += NT) {
          const int r = i / Q, c4 = i % Q;
          float4 v = *reinterpret_cast<const float4*>(DM + r * Lay::LDM + c4 * 4);
          if (KIND == NODE_BLOCK && pass == 0) {
            const float4 d = reinterpret_cast<const float4*>(a.dm + (row0 + r) * L)[c4];
            v.x += d.x;
            v.y += d.y;
            v.z += d.z;
            v.w += d.w;
          }
          reinterpret_cast<float4*>(dst + (row0 + r) * L)[c4] = v;
        }
      }
    }
    __syncthreads();
  }
  // per-workgroup vector partials: [db_0 .. db_{D-1}, gamma, beta]
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  if (wave_has_cols && (threadIdx.x & 63) < 16) {
#pragma unroll
    for (int j = 0; j < D - 1; ++j)
#pragma unroll
      for (int nn = 0; nn < NBW; ++nn) vp[j * L + (wave * NBW + nn) * 16 + (threadIdx.x & 15)] = g_bh[j][nn];
  }
  const int off_last = (D - 1) * L;
  if (tid < nout_last) vp[off_last + tid] = g_blast;
  if constexpr (S::LN) {
    if (tid < L) {
      vp[off_last + L + tid] = g_gamma;
      vp[off_last + 2 * L + tid] = g_beta;
    }
  }
}

// ---------------------------------------------------------- edge kernels ---
// LDS of the edge kernels for TE rows: A holds [e | v_s | v_r] (storage type);
// in the backward pass the same bytes then hold xhat (fp32, 4L bytes per row)
// followed by the gradient in storage type.  B, C: hidden activations.  D:
// fp32 gradient / output staging.
template <class P, int L, int D, int TE>
struct EdgeLds {
  using T = typename P::T;
  static constexpr int LDA = 3 * L + P::PAD;                    // storage-type elements
  static constexpr int ROWB = LDA * (int)sizeof(T);             // bytes per A row
  static constexpr int LDY = ROWB / 4;                          // fp32 stride over A rows
  static constexpr int Y_OFF_F = L * (int)sizeof(T) / 4;        // forward: Y after e (fp32 index)
  static constexpr int DY_OFF = 4 * L / (int)sizeof(T);         // backward: DY after xhat (T index)
  static constexpr int LDH = L + P::PAD;
  static constexpr int LDM = L + 4;
  static constexpr int AB = TE * ROWB;
  static constexpr int HB = TE * LDH * (int)sizeof(T);
  static constexpr int OFF_B = rup(AB, 16);
  static constexpr int OFF_C = OFF_B + HB;
  static constexpr int OFF_D = OFF_C + (D == 3 ? HB : 0);
  static constexpr int OFF_META = OFF_D + TE * LDM * 4;            // backward: rr, ss, mask, rstd
  static constexpr int END = OFF_META + TE * 12 + 16;
  static constexpr int END_F = OFF_D + TE * 8 + 16;                  // forward: rr, ss, mask after B/C
};

template <class P, int L, int D>
struct EdgeTE {
  static constexpr int value = EdgeLds<P, L, D, 64>::END <= LDS_MAX   ? 64
                               : EdgeLds<P, L, D, 32>::END <= LDS_MAX ? 32
                                                                      : 16;
};

// Backward sub-tiles are capped at 32 rows: the smaller LDS footprint lets
// two workgroups share a CU, which hides more gather latency than the larger
// tile saves in weight-fragment reloads.
template <class P, int L, int D>
struct EdgeTEB {
  static constexpr int value = EdgeTE<P, L, D>::value > 32 ? 32 : EdgeTE<P, L, D>::value;
};

// Per-row metadata of a sub-tile in LDS: receiver and sender local ids, and a
// bit mask of the rows that end their receiver's segment.
struct EdgeMeta {
  int32_t* rr;
  int32_t* ss;
  unsigned long long* last;
};

// Loads a sub-tile's metadata into LDS (receiver and sender ids of its TE
// rows, and which rows end a receiver segment), then synchronises.
template <int TE>
__device__ __forceinline__ void stage_meta(EdgeMeta mt, const int32_t* erecv, const int32_t* send, int64_t sb,
                                           int n, int64_t e1) {
  const int tid = threadIdx.x;
  if (tid < 64) {
    int32_t r = -1, sd = 0;
    bool l = false;
    if (tid < n) {
      const int64_t e = sb + tid;
      r = erecv[e];
      sd = send[e];
      l = (e + 1 == e1) || erecv[e + 1] != r;
    }
    const unsigned long long m = __ballot(l);
    if (tid < TE) {
      mt.rr[tid] = r;
      mt.ss[tid] = sd;
    }
    if (tid == 0) *mt.last = m;
  }
  __syncthreads();
}

// Gathers the rows [e | v_s | v_r] of a sub-tile whose metadata is in LDS.
// Every row load of this thread is issued before any is stored, so the
// gather costs one memory latency, not one per row.  No barrier at the end.
template <class P, int L, int TE, int LDA>
__device__ __forceinline__ void gather_rows(typename P::T* A, EdgeMeta mt, const typename P::T* Ein, const float* V,
                                            const float* H, const void* V16, int64_t n_owned, int64_t sb, int n) {
  using T = typename P::T;
  const int tid = threadIdx.x;
  constexpr int E16 = 16 / sizeof(T);
  constexpr int CPR = L / E16;                   // 16-byte chunks per e row
  if constexpr (sizeof(T) == 2) {
    // bf16: e^k rows and the bf16 copy of the node rows, 16-byte chunks
    const T* V16t = reinterpret_cast<const T*>(V16);
    constexpr int IT = (TE * 3 * CPR + NT - 1) / NT;
    uint4 buf[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int i = tid + j * NT, r = i / (3 * CPR), rem = i % (3 * CPR), part = rem / CPR;
      const int c = (rem % CPR) * E16;
      buf[j] = make_uint4(0, 0, 0, 0);
      if (i < TE * 3 * CPR && r < n) {
        const T* src = part == 0 ? Ein + (sb + r) * L : V16t + (int64_t)(part == 1 ? mt.ss[r] : mt.rr[r]) * L;
        buf[j] = *reinterpret_cast<const uint4*>(src + c);
      }
    }
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int i = tid + j * NT, r = i / (3 * CPR), rem = i % (3 * CPR), part = rem / CPR;
      const int c = (rem % CPR) * E16;
      if (i < TE * 3 * CPR) *reinterpret_cast<uint4*>(A + r * LDA + part * L + c) = buf[j];
    }
    return;
  }
  constexpr int IE = (TE * CPR + NT - 1) / NT;
  constexpr int Q = L / 4;                       // float4 per node row
  constexpr int IV = (TE * 2 * Q + NT - 1) / NT;
  uint4 ev[IE];
  float4 vv[IV];
#pragma unroll
  for (int j = 0; j < IE; ++j) {
    const int i = tid + j * NT, r = i / CPR, c = (i % CPR) * E16;
    ev[j] = make_uint4(0, 0, 0, 0);
    if (i < TE * CPR && r < n) ev[j] = *reinterpret_cast<const uint4*>(Ein + (sb + r) * L + c);
  }
#pragma unroll
  for (int j = 0; j < IV; ++j) {
    const int i = tid + j * NT, r = i / (2 * Q), rem = i % (2 * Q), sside = rem / Q, c4 = rem % Q;
    vv[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < TE * 2 * Q && r < n) {
      const float* src;
      if (sside == 0) {
        const int64_t snd = mt.ss[r];
        src = snd < n_owned ? V + snd * L : H + (snd - n_owned) * L;
      } else {
        src = V + (int64_t)mt.rr[r] * L;
      }
      vv[j] = reinterpret_cast<const float4*>(src)[c4];
    }
  }
#pragma unroll
  for (int j = 0; j < IE; ++j) {
    const int i = tid + j * NT, r = i / CPR, c = (i % CPR) * E16;
    if (i < TE * CPR) *reinterpret_cast<uint4*>(A + r * LDA + c) = ev[j];
  }
#pragma unroll
  for (int j = 0; j < IV; ++j) {
    const int i = tid + j * NT, r = i / (2 * Q), rem = i % (2 * Q), sside = rem / Q, c4 = rem % Q;
    if (i < TE * 2 * Q) st4<P>(A + r * LDA + (1 + sside) * L + c4 * 4, vv[j]);
  }
}

// Metadata, then rows: the whole staging of a sub-tile (no barrier at the end).
template <class P, int L, int TE, int LDA>
__device__ __forceinline__ void stage_edges(typename P::T* A, EdgeMeta mt, const int32_t* erecv,
                                            const int32_t* send, const typename P::T* Ein, const float* V,
                                            const float* H, const void* V16, int64_t n_owned, int64_t sb, int n,
                                            int64_t e1) {
  stage_meta<TE>(mt, erecv, send, sb, n, e1);
  gather_rows<P, L, TE, LDA>(A, mt, Ein, V, H, V16, n_owned, sb, n);
}

// Ordered running sum over the rows of a sub-tile for column c: adds rows
// 0..n-1 of M (fp32 or storage type, row stride ld) to `run`; at each row
// that ends a receiver segment, hands the segment's total to emit(receiver,
// total) and restarts.  The running value carries into the next sub-tile of
// the unit.
template <int TE, class MT, class Emit>
__device__ __forceinline__ void segment_sums(const MT* M, int ld, int n, int c, EdgeMeta mt, float& run,
                                             Emit emit) {
  const unsigned long long mask = *mt.last;
#pragma unroll 8
  for (int r = 0; r < TE; ++r) {
    if (r < n) {
      run += to_f(M[r * ld + c]);
      if ((mask >> r) & 1ull) {
        emit(mt.rr[r], run);
        run = 0.f;
      }
    }
  }
}

// Zeroes `width` fp32 columns of the rows of receivers in [r0, r1) that have no
// edges (their ordered sums are empty).
__device__ __forceinline__ void zero_empty_receivers(const int32_t* row_ptr, int64_t r0, int64_t r1, float* dst,
                                                     int L) {
  for (int64_t r = r0 + threadIdx.x; r < r1; r += NT)
    if (row_ptr[r] == row_ptr[r + 1])
      for (int c = 0; c < L; c += 4) *reinterpret_cast<float4*>(dst + r * L + c) = make_float4(0.f, 0.f, 0.f, 0.f);
}

// Waves per SIMD the streaming edge kernels are compiled for: two where two
// workgroups fit the LDS (the edge gather's latency needs them more than the
// products need registers); at l = 256 one workgroup fills the LDS, and one
// wave per SIMD may use the accumulator registers too instead of spilling.
template <int L>
struct EdgeWpe {
  static constexpr int value = L >= 256 ? 1 : 2;
};

template <int P_, int L, int D>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(EdgeWpe<L>::value))) void edge_fwd_kernel(EdgeFwdArgs a) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  constexpr int TE = EdgeTE<P, L, D>::value;
  using Lay = EdgeLds<P, L, D, TE>;
  constexpr int MB = TE / 16;
  constexpr int NBW = L / 16 / NW > 0 ? L / 16 / NW : 1;
  extern __shared__ __align__(16) unsigned char lds[];
  T* A = reinterpret_cast<T*>(lds);
  T* HB = reinterpret_cast<T*>(lds + Lay::OFF_B);
  T* HC = reinterpret_cast<T*>(lds + Lay::OFF_C);
  float* Y = reinterpret_cast<float*>(lds) + Lay::Y_OFF_F;
  EdgeMeta mt;
  mt.rr = reinterpret_cast<int32_t*>(lds + Lay::OFF_D);
  mt.ss = mt.rr + TE;
  mt.last = reinterpret_cast<unsigned long long*>(mt.ss + TE);
  const int wave = threadIdx.x >> 6, tid = threadIdx.x;
  const bool wave_has_cols = wave * NBW * 16 < L;
  const T* Ein = reinterpret_cast<const T*>(a.Ein);
  T* Eout = reinterpret_cast<T*>(a.Eout);
  constexpr int NK1 = 3 * L / P::KG, NKH = L / P::KG;

  for (TileIter it(*a.n_units); it.valid(); it.next()) {
    const int64_t r0 = a.unit_r[it.t], r1 = a.unit_r[it.t + 1];
    const int64_t e0 = a.row_ptr[r0], e1 = a.row_ptr[r1];
    zero_empty_receivers(a.row_ptr, r0, r1, a.agg, L);
    float run = 0.f;  // running receiver sum of column tid
    for (int64_t sb = e0; sb < e1; sb += TE) {
      const int n = (int)(e1 - sb < TE ? e1 - sb : TE);
      stage_edges<P, L, TE, Lay::LDA>(A, mt, a.erecv, a.send, Ein, a.V, a.H, a.V16, a.n_owned, sb, n, e1);
      __syncthreads();
      {
        floatx4 acc[MB][NBW];
        if (wave_has_cols) {
          wave_gemm_k<P, MB, NBW, NK1>(A, Lay::LDA, a.mlp.lin[0].wf, wave * NBW, acc);
          store_acc<P, MB, NBW, true>(acc, wave * NBW, a.mlp.lin[0].b, L, HB, Lay::LDH);
        }
      }
      __syncthreads();
      // kept for the backward (HB is read-only until the next sub-tile)
      if (a.hid_out) store_rows(reinterpret_cast<T*>(a.hid_out) + sb * L, HB, Lay::LDH, n, L);
      const T* hin = HB;
      if constexpr (D == 3) {
        floatx4 acc[MB][NBW];
        if (wave_has_cols) {
          wave_gemm_k<P, MB, NBW, NKH>(HB, Lay::LDH, a.mlp.lin[1].wf, wave * NBW, acc);
          store_acc<P, MB, NBW, true>(acc, wave * NBW, a.mlp.lin[1].b, L, HC, Lay::LDH);
        }
        __syncthreads();
        hin = HC;
      }
      {
        floatx4 acc[MB][NBW];
        if (wave_has_cols) {
          wave_gemm_k<P, MB, NBW, NKH>(hin, Lay::LDH, a.mlp.lin[D - 1].wf, wave * NBW, acc);
          store_acc<P, MB, NBW, false>(acc, wave * NBW, a.mlp.lin[D - 1].b, L, Y, Lay::LDY);
        }
      }
      __syncthreads();
      ln_rows<TE, L>(Y, Lay::LDY, a.eps, a.mlp.gamma, a.mlp.beta);
      __syncthreads();
      if (Eout) {
        // e^{k+1} = e^k + m, 16 bytes of output per thread
        constexpr int E16 = 16 / sizeof(T);
        constexpr int CPR = L / E16;
        for (int i = tid; i < n * CPR; i += NT) {
          const int r = i / CPR, c = (i % CPR) * E16;
          T o[E16];
#pragma unroll
          for (int j = 0; j < E16; ++j) o[j] = P::cvt(P::tof(A[r * Lay::LDA + c + j]) + Y[r * Lay::LDY + c + j]);
          *reinterpret_cast<uint4*>(Eout + (sb + r) * L + c) = *reinterpret_cast<const uint4*>(o);
        }
      }
      if (tid < L)
        segment_sums<TE>(Y, Lay::LDY, n, tid, mt, run,
                         [&](int32_t r, float v) { a.agg[(int64_t)r * L + tid] = v; });
      __syncthreads();
    }
  }
}

// LDS of the edge backward kernel for TE rows: A holds [e | v_s | v_r]
// (storage type) for the recompute and then the gradients: dy at columns
// 0..L, dz of the hidden layers at L.. and 2L..; B, C: hidden activations;
// the sub-tile metadata; slots for cross-wave row reductions.
template <class P, int L, int D, int TE>
struct EdgeBwdLds {
  using T = typename P::T;
  static constexpr int LDA = 3 * L + P::PAD;
  static constexpr int LDH = L + P::PAD;
  static constexpr int HB = TE * LDH * (int)sizeof(T);
  static constexpr int OFF_B = rup(TE * LDA * (int)sizeof(T), 16);
  static constexpr int OFF_C = OFF_B + HB;
  static constexpr int OFF_META = OFF_C + (D == 3 ? HB : 0);
  static constexpr int OFF_RED = OFF_META + rup(TE * 8 + 8, 16);
  static constexpr int END = OFF_RED + 4 * NW * TE * 4;
};

// Backward of one block's edge half with the forward recomputed in the tile.
// Per edge: dm = de^{k+1} + dagg[receiver]; LayerNorm backward; the MLP's
// backward down to dz_0, the gradient at the first Linear's output; then
// de^k = de^{k+1} + dz_0 W_1[:, e-block].  The sender and receiver blocks of
// W_1 are the same for every edge, so their products are taken per node
// later (input_grad_kernel): here each receiver's sum of dz_0 (in the
// precision that feeds the products) overwrites its dagg row once the last of
// its edges is done, and receivers without edges get a zero row.  dz_0, the
// LN-backward output and the hidden activations go to HBM for the weight
// gradients; bias / gamma / beta gradients are per-lane column partials over
// the workgroup's rows, written once at the end.
// How the edge backward obtains the first Linear's ReLU output h_1: recompute
// it from the gathered [e | v_s | v_r] rows, or read the forward's copy.  One
// instantiation per way keeps the other's registers out.
enum { BWD_GATHER = 0, BWD_STASH = 1 };

template <int P_, int L, int D, int MODE>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(EdgeWpe<L>::value))) void edge_bwd_kernel(EdgeBwdArgs a) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  constexpr int TE = EdgeTEB<P, L, D>::value;
  using Lay = EdgeBwdLds<P, L, D, TE>;
  constexpr int MB = TE / 16;
  constexpr int NBW = L / 16 / NW;
  static_assert(NBW >= 1 && L % (16 * NW) == 0, "latent width must be a multiple of 64");
  constexpr int NK1 = 3 * L / P::KG, NKH = L / P::KG;
  extern __shared__ __align__(16) unsigned char lds[];
  T* A = reinterpret_cast<T*>(lds);
  T* HB = reinterpret_cast<T*>(lds + Lay::OFF_B);
  T* HC = reinterpret_cast<T*>(lds + Lay::OFF_C);
  EdgeMeta mt;
  mt.rr = reinterpret_cast<int32_t*>(lds + Lay::OFF_META);
  mt.ss = mt.rr + TE;
  mt.last = reinterpret_cast<unsigned long long*>(mt.ss + TE);
  float* red = reinterpret_cast<float*>(lds + Lay::OFF_RED);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, tid = threadIdx.x;
  const int nb0 = wave * NBW;
  const T* Ein = reinterpret_cast<const T*>(a.Ein);

  float gam[NBW], blast[NBW];
#pragma unroll
  for (int n = 0; n < NBW; ++n) {
    const int col = (nb0 + n) * 16 + acc_col();
    gam[n] = a.mlp.gamma[col];
    blast[n] = a.mlp.lin[D - 1].b[col];
  }
  // column partials over this lane's rows: gamma, beta, last bias, hidden biases
  float pg[NBW], pb[NBW], pl[NBW], ph[2][NBW];
#pragma unroll
  for (int n = 0; n < NBW; ++n) pg[n] = pb[n] = pl[n] = ph[0][n] = ph[1][n] = 0.f;

  // the work units of the receiver range [r_lo, r_hi) (unit boundaries fall on it)
  int u_lo, u_hi;
  {
    const int nu = *a.n_units;
    auto lower = [&](int64_t r) {
      int lo = 0, hi = nu;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (a.unit_r[mid] < r) lo = mid + 1;
        else hi = mid;
      }
      return lo;
    };
    u_lo = lower(a.r_lo);
    u_hi = lower(a.r_hi);
  }
  for (TileIter it(u_hi - u_lo, u_lo); it.valid(); it.next()) {
    const int64_t r0 = a.unit_r[it.t], r1 = a.unit_r[it.t + 1];
    const int64_t e0 = a.row_ptr[r0], e1 = a.row_ptr[r1];
    zero_empty_receivers(a.row_ptr, r0, r1, a.dagg, L);
    float run = 0.f;  // running receiver sum of dz_0, column tid
    for (int64_t sb = e0; sb < e1; sb += TE) {
      const int n = (int)(e1 - sb < TE ? e1 - sb : TE);
      stage_meta<TE>(mt, a.erecv, a.send, sb, n, e1);
      // dm = de^{k+1} + dagg[receiver] in accumulator layout, issued before
      // the row gather so that both latencies overlap
      float de[MB][NBW][4], da[MB][NBW][4];
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m * 16 + acc_row(r);
          const bool ok = row < n;
          const int64_t rv = ok ? (int64_t)mt.rr[row] : 0;
#pragma unroll
          for (int nn = 0; nn < NBW; ++nn) {
            const int col = (nb0 + nn) * 16 + acc_col();
            de[m][nn][r] = (ok && a.de_next) ? P::tof(reinterpret_cast<const T*>(a.de_next)[(sb + row) * L + col]) : 0.f;
            da[m][nn][r] = ok ? a.dagg[rv * L + col] : 0.f;
          }
        }
      if constexpr (MODE == BWD_STASH) {
        // the forward's first-Linear ReLU output (rows past n zero: they
        // carry dm = 0 and contribute nothing)
        constexpr int E16 = 16 / sizeof(T);
        constexpr int CPR = L / E16;
        const T* hsrc = reinterpret_cast<const T*>(a.hid_in) + sb * L;
        for (int i = tid; i < TE * CPR; i += NT) {
          const int r = i / CPR, c = (i % CPR) * E16;
          uint4 v = make_uint4(0, 0, 0, 0);
          if (r < n) v = *reinterpret_cast<const uint4*>(hsrc + (int64_t)r * L + c);
          *reinterpret_cast<uint4*>(HB + r * Lay::LDH + c) = v;
        }
      } else {
        gather_rows<P, L, TE, Lay::LDA>(A, mt, Ein, a.V, a.H, a.V16, a.n_owned, sb, n);
        __syncthreads();
        // recompute the forward: hidden activations, then the LN input
        floatx4 acc[MB][NBW];
        wave_gemm_k<P, MB, NBW, NK1>(A, Lay::LDA, a.mlp.lin[0].wf, nb0, acc);
        store_acc<P, MB, NBW, true>(acc, nb0, a.mlp.lin[0].b, L, HB, Lay::LDH);
      }
      __syncthreads();
      const T* hin = HB;
      if constexpr (D == 3) {
        floatx4 acc[MB][NBW];
        wave_gemm_k<P, MB, NBW, NKH>(HB, Lay::LDH, a.mlp.lin[1].wf, nb0, acc);
        store_acc<P, MB, NBW, true>(acc, nb0, a.mlp.lin[1].b, L, HC, Lay::LDH);
        __syncthreads();
        hin = HC;
      }
      floatx4 y[MB][NBW];
      wave_gemm_k<P, MB, NBW, NKH>(hin, Lay::LDH, a.mlp.lin[D - 1].wf, nb0, y);
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int nn = 0; nn < NBW; ++nn)
#pragma unroll
          for (int r = 0; r < 4; ++r) y[m][nn][r] += blast[nn];
      float rs[MB][4];
      ln_tile<MB, NBW, L>(y, a.eps, red, red + NW * TE, rs);  // y now holds xhat
      // LayerNorm backward: dy = rstd (dm g - mean(dm g) - xhat mean(dm g xhat))
      float s2[2][MB][4];
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float s1 = 0.f, sx = 0.f;
#pragma unroll
          for (int nn = 0; nn < NBW; ++nn) {
            const float dm = da[m][nn][r] + de[m][nn][r];
            const float d = dm * gam[nn];
            s1 += d;
            sx += d * y[m][nn][r];
            pg[nn] += dm * y[m][nn][r];
            pb[nn] += dm;
          }
          s2[0][m][r] = s1;
          s2[1][m][r] = sx;
        }
      row_totals<2, MB>(s2, red + 2 * NW * TE);
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m * 16 + acc_row(r);
          const float m1 = s2[0][m][r] / L, m2 = s2[1][m][r] / L;
#pragma unroll
          for (int nn = 0; nn < NBW; ++nn) {
            const int col = (nb0 + nn) * 16 + acc_col();
            const float dm = da[m][nn][r] + de[m][nn][r];
            const float dy = rs[m][r] * (dm * gam[nn] - m1 - y[m][nn][r] * m2);
            pl[nn] += dy;
            A[row * Lay::LDA + col] = P::cvt(dy);
          }
        }
      __syncthreads();
      store_rows(reinterpret_cast<T*>(a.delta[D - 1]) + (sb - a.e_base) * L, A, Lay::LDA, n, L);
      if constexpr (MODE != BWD_STASH) store_rows(reinterpret_cast<T*>(a.hid[0]) + (sb - a.e_base) * L, HB, Lay::LDH, n, L);
      if constexpr (D == 3) store_rows(reinterpret_cast<T*>(a.hid[1]) + (sb - a.e_base) * L, HC, Lay::LDH, n, L);
      // hidden layers: dz_{j-1} = (dz_j W_j) * [h_{j-1} > 0], into A column block D-j
#pragma unroll
      for (int j = D - 1; j >= 1; --j) {
        const T* din = A + (D - 1 - j) * L;
        T* dout = A + (D - j) * L;
        const T* hprev = (j == 2) ? HC : HB;
        floatx4 acc[MB][NBW];
        wave_gemm_k<P, MB, NBW, NKH>(din, Lay::LDA, a.mlp.lin[j].wb, nb0, acc);
#pragma unroll
        for (int nn = 0; nn < NBW; ++nn)
#pragma unroll
          for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = m * 16 + acc_row(r), col = (nb0 + nn) * 16 + acc_col();
              const float v = P::tof(hprev[row * Lay::LDH + col]) > 0.f ? acc[m][nn][r] : 0.f;
              ph[j - 1][nn] += v;
              dout[row * Lay::LDA + col] = P::cvt(v);
            }
        __syncthreads();
        store_rows(reinterpret_cast<T*>(a.delta[j - 1]) + (sb - a.e_base) * L, dout, Lay::LDA, n, L);
      }
      // edge-stream gradient: de^k = de^{k+1} + dz_0 W_1[:, e-block]
      const T* dz0 = A + (D - 1) * L;
      {
        floatx4 acc[MB][NBW];
        wave_gemm_k<P, MB, NBW, NKH>(dz0, Lay::LDA, a.mlp.lin[0].wb, nb0, acc);
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = m * 16 + acc_row(r);
            if (row < n) {
#pragma unroll
              for (int nn = 0; nn < NBW; ++nn)
                reinterpret_cast<T*>(a.de_out)[(sb + row) * L + (nb0 + nn) * 16 + acc_col()] =
                    P::cvt(acc[m][nn][r] + de[m][nn][r]);
            }
          }
      }
      // receiver sums of dz_0, ascending edge order
      if (tid < L)
        segment_sums<TE>(dz0, Lay::LDA, n, tid, mt, run,
                         [&](int32_t r, float v) { a.dagg[(int64_t)r * L + tid] = v; });
      __syncthreads();
    }
  }
  // column partials: the four 16-lane groups of a column, then one writer lane
#pragma unroll
  for (int nn = 0; nn < NBW; ++nn) {
    float* v[5] = {&pg[nn], &pb[nn], &pl[nn], &ph[0][nn], &ph[1][nn]};
#pragma unroll
    for (int q = 0; q < 5; ++q) {
      float x = *v[q];
      x += __shfl_xor(x, 16, 64);
      x += __shfl_xor(x, 32, 64);
      *v[q] = x;
    }
  }
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  if (lane < 16) {
    const int off_last = (D - 1) * L;
#pragma unroll
    for (int nn = 0; nn < NBW; ++nn) {
      const int col = (nb0 + nn) * 16 + lane;
#pragma unroll
      for (int j = 0; j < D - 1; ++j) vp[j * L + col] = ph[j][nn];
      vp[off_last + col] = pl[nn];
      vp[off_last + L + col] = pg[nn];
      vp[off_last + 2 * L + col] = pb[nn];
    }
  }
}

// ------------------------------------------------ row-split edge kernels ---
// bf16, latent 64 or 128.  The first Linear of the edge MLP acts on
// [e | v_s | v_r]; its sender and receiver blocks are applied per node once
// per block (node_proj_kernel: P[n] = [W_s v_n | W_r v_n], fp32), so per edge
// z_1 = W_e e + P_s[s] + P_r[r] + b_1 and the per-edge weights shrink to
// L x L matrices.  Those sit in LDS, shared by the workgroup's waves, and
// every wave works alone on 16-edge tiles of its own receiver-aligned edge
// range: A operands come straight from HBM in MFMA fragment order, row-wise
// quantities (LayerNorm statistics, segment sums) stay inside the wave, and
// there is no barrier in the edge loop, so one wave's memory latency hides
// behind the others' products.  A wave-private LDS scratch turns
// accumulator tiles back into row order (operands of the next product,
// coalesced row stores).

constexpr int RS_NWV = 8;              // waves per workgroup
constexpr int RS_NTH = 64 * RS_NWV;
constexpr int RS_GRID = 256;           // one workgroup per compute unit; a multiple of 8

// bf16 / fp32 element index of (row, col) in a 16-row scratch tile of width
// L whose 16-byte chunks are XOR-swizzled by row (conflict-free both for
// accumulator-order writes and for fragment / row-order reads).
template <int L>
__device__ __forceinline__ int rs_sw16(int row, int col) {
  constexpr int M = (L / 8 < 16 ? L / 8 : 16) - 1;
  return row * L + ((((col >> 3) ^ (row & M))) << 3) + (col & 7);
}
template <int L>
__device__ __forceinline__ int rs_sw32(int row, int col) {
  constexpr int M = (L / 4 < 16 ? L / 4 : 16) - 1;
  return row * L + ((((col >> 2) ^ (row & M))) << 2) + (col & 3);
}

// acc[cb] = sum over k-groups of A[kg] x B[cb][kg]: one 16-row tile, every
// 16-column block cb, B fragments in LDS ([cb][kg][lane], 16 bytes each).
template <int NB, int NKG>
__device__ __forceinline__ void rs_gemm(const uint4 (&A)[NKG], const uint4* Bl, floatx4 (&acc)[NB], int lane) {
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kg = 0; kg < NKG; ++kg)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) PBF16::mma(acc[cb], A[kg], Bl[(cb * NKG + kg) * 64 + lane]);
}

// Copies nb 16-column blocks x nkg k-groups of packed fragments (source
// block stride src_nkg k-groups, first k-group kg0) into LDS, all threads.
__device__ __forceinline__ void rs_copy_frags(uint4* dst, const uint4* __restrict__ src, int nb, int nkg, int src_nkg,
                                              int kg0) {
  const int total = nb * nkg * 64;
  for (int i = threadIdx.x; i < total; i += blockDim.x) {
    const int cb = i / (nkg * 64), kg = (i / 64) % nkg, ln = i % 64;
    dst[i] = src[((size_t)cb * src_nkg + kg0 + kg) * 64 + ln];
  }
}

// The wave's index in its workgroup, as a wave-uniform (scalar) value.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// A wave-uniform value held in scalar registers.
__device__ __forceinline__ int64_t rs_uniform(int64_t x) {
  const uint64_t u = (uint64_t)x;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Receiver range of wave w (of W waves in total) within [lo_r, hi_r):
// receiver-aligned, about E / W edges each; the waves of one XCD
// (blockIdx % 8) get neighbouring ranges.
__device__ __forceinline__ void rs_range(const int32_t* __restrict__ row_ptr, int64_t lo_r, int64_t hi_r, int64_t& r0,
                                         int64_t& r1) {
  const int G = gridDim.x, b = blockIdx.x, nwv = blockDim.x >> 6, wave = wave_id();
  const int64_t W = (int64_t)G * nwv;
  const int64_t q = ((int64_t)(b & 7) * (G >> 3) + (b >> 3)) * nwv + wave;
  const int64_t e0 = row_ptr[lo_r], E = row_ptr[hi_r] - e0;
  auto find = [&](int64_t target) {  // first receiver r >= lo_r with row_ptr[r] >= target
    int64_t lo = lo_r, hi = hi_r;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (row_ptr[mid] >= target) hi = mid;
      else lo = mid + 1;
    }
    return lo;
  };
  r0 = q == 0 ? lo_r : find(e0 + E * q / W);
  r1 = q + 1 == W ? hi_r : find(e0 + E * (q + 1) / W);
}

// Zeroes the rows (width L) of the receivers in [r0, r1) without edges (one
// wave, a lane per receiver).
__device__ __forceinline__ void rs_zero_empty(const int32_t* __restrict__ row_ptr, int64_t r0, int64_t r1, float* dst,
                                              int L) {
  const int lane = threadIdx.x & 63;
  for (int64_t r = r0 + lane; r < r1; r += 64)
    if (row_ptr[r] == row_ptr[r + 1])
      for (int c = 0; c < L; c += 4) *reinterpret_cast<float4*>(dst + r * L + c) = make_float4(0.f, 0.f, 0.f, 0.f);
}

// ----------------------------------------------------------------- T form ---
// The row-split edge kernels and node_proj_kernel compute every product
// transposed, Y^T = W X^T: weight fragments are the MFMA A operand and a
// 16-row tile of activations the B operand (lane (e, q) = (lane & 15,
// lane >> 4) supplies row e, k-slots 8 q ..).  Lane (e, q) of the
// accumulator tile then holds output columns 16 cb + 4 q + r (every 16-column
// block cb, r = 0..3) of row e.  Three things follow.  Rounded to bf16, the
// accumulators of one product are the B operand of the next as they stand:
// for k-group kg lane (e, q) has columns 32 kg + 16 h + 4 q + r (h = 0, 1),
// which the next weight matrix's fragments match once their k-slots are
// permuted the same way (rt_copy_frags).  A row's LayerNorm statistics are a
// per-lane sum plus a sum over the four 16-lane groups (two lane-swap
// instructions).  Column sums over a tile's rows are a reduce-scatter across
// the 16 lanes of a group (DPP).  Rows in memory keep the plain column order:
// a lane reads or writes 4 consecutive columns per 16-column block.

// One 16-edge tile's metadata, every lane for its row e = lane & 15: the
// edge's receiver, sender and the next edge's receiver (-1 past the range
// end); the mask has bit j (j < 16) set where row j ends a receiver segment.
// The loads are issued one tile ahead (rt_meta_load) and turned into the
// mask when the tile starts (rt_meta_make), so no tile waits for them.
struct RsMeta {
  int32_t r, s;
  unsigned long long last;
};
struct RsMetaRaw {
  int32_t r, s, rn;
};
__device__ __forceinline__ RsMetaRaw rt_meta_load(const int32_t* __restrict__ erecv, const int32_t* __restrict__ send,
                                                  int64_t sb, int64_t e1) {
  const int e = threadIdx.x & 15;
  RsMetaRaw w{-1, 0, -1};
  if (sb + e < e1) {
    w.r = erecv[sb + e];
    w.s = send[sb + e];
    if (sb + e + 1 < e1) w.rn = erecv[sb + e + 1];
  }
  return w;
}
__device__ __forceinline__ RsMeta rt_meta_make(const RsMetaRaw& w) {
  RsMeta mt{w.r, w.s, 0};
  mt.last = __ballot(w.r >= 0 && w.rn != w.r);
  return mt;
}

// Like rs_copy_frags, with the eight k-slots of every fragment reordered so
// that slot j of lane group q pairs with k = 32 kg + 16 (j / 4) + 4 q + j % 4:
// its low half comes from lane group q / 2, its high half from 2 + q / 2,
// slots 4 (q % 2) .. of each.
__device__ __forceinline__ void rt_copy_frags(uint4* dst, const uint4* __restrict__ src, int nb, int nkg, int src_nkg,
                                              int kg0) {
  const int total = nb * nkg * 64;
  for (int i = threadIdx.x; i < total; i += blockDim.x) {
    const int cb = i / (nkg * 64), kg = (i / 64) % nkg, ln = i % 64, q = ln >> 4, c = ln & 15;
    const uint2* s = reinterpret_cast<const uint2*>(src + ((size_t)cb * src_nkg + kg0 + kg) * 64);
    const uint2 lo = s[(c + 16 * (q >> 1)) * 2 + (q & 1)];
    const uint2 hi = s[(c + 16 * (2 + (q >> 1))) * 2 + (q & 1)];
    dst[i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
}

// acc[cb] = sum over k-groups of W[cb][kg] (LDS, [cb][kg][lane]) x X[kg].
template <int NB, int NKG>
__device__ __forceinline__ void rt_gemm(const uint4* Wl, const uint4 (&X)[NKG], floatx4 (&acc)[NB], int lane) {
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kg = 0; kg < NKG; ++kg)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) PBF16::mma(acc[cb], Wl[(cb * NKG + kg) * 64 + lane], X[kg]);
}

// Two fp32 values -> two bf16 (round to nearest even, one conversion instruction).
__device__ __forceinline__ uint32_t bf_pack(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Accumulator-order values -> bf16 B operands of the next product.
template <int NB>
__device__ __forceinline__ void rt_frags(const float (&v)[NB][4], uint4 (&f)[NB / 2]) {
#pragma unroll
  for (int kg = 0; kg < NB / 2; ++kg)
    f[kg] = make_uint4(bf_pack(v[2 * kg][0], v[2 * kg][1]), bf_pack(v[2 * kg][2], v[2 * kg][3]),
                       bf_pack(v[2 * kg + 1][0], v[2 * kg + 1][1]), bf_pack(v[2 * kg + 1][2], v[2 * kg + 1][3]));
}

// T-order bf16 of one k-group -> plain order.  In: lane group q holds
// columns 32 kg + 4 q .. +3 (x, y) and 32 kg + 16 + 4 q .. +3 (z, w).  Out:
// columns 32 kg + 8 q .. +7, one 16-byte row chunk.  A lane swap between the
// group pairs (0, 1) <-> (2, 3), then one between groups 0 <-> 1 and 2 <-> 3.
__device__ __forceinline__ uint4 rt_to_plain(const uint4 f) {
  const auto s0 = __builtin_amdgcn_permlane32_swap(f.x, f.z, false, false);
  const auto s1 = __builtin_amdgcn_permlane32_swap(f.y, f.w, false, false);
  const auto t0 = __builtin_amdgcn_permlane16_swap(s0[0], s0[1], false, false);
  const auto t1 = __builtin_amdgcn_permlane16_swap(s1[0], s1[1], false, false);
  return make_uint4(t0[0], t1[0], t0[1], t1[1]);
}
// Inverse of rt_to_plain (both swaps are involutions, applied in reverse).
__device__ __forceinline__ uint4 rt_from_plain(const uint4 p) {
  const auto t0 = __builtin_amdgcn_permlane16_swap(p.x, p.z, false, false);
  const auto t1 = __builtin_amdgcn_permlane16_swap(p.y, p.w, false, false);
  const auto s0 = __builtin_amdgcn_permlane32_swap(t0[0], t0[1], false, false);
  const auto s1 = __builtin_amdgcn_permlane32_swap(t1[0], t1[1], false, false);
  return make_uint4(s0[0], s1[0], s0[1], s1[1]);
}

// The values of rt_frags -> one plain-order bf16 row, 16 bytes per lane and
// k-group.  All lanes take part in the swaps; only lanes with ok store.
// A stored bf16 ReLU output row as read (plain order: lane (e, q) holds its
// row's k-slots kg * 32 + 8 q ..) -> T-order fragments, and the ReLU mask
// their signs give: bit cb * 4 + r is set where the value is positive.
// rt_load_relu reads the row as well.
template <int NKH>
__device__ __forceinline__ void rt_relu_frags(const uint4 (&raw)[NKH], uint4 (&hf)[NKH], uint32_t& mask) {
#pragma unroll
  for (int kg = 0; kg < NKH; ++kg) {
    hf[kg] = rt_from_plain(raw[kg]);
    const uint32_t w[4] = {hf[kg].x, hf[kg].y, hf[kg].z, hf[kg].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // dword i: block 2 kg + i / 2, rows r = 2 (i % 2) .. + 1
      const int cb = 2 * kg + i / 2, r = 2 * (i % 2);
      mask |= ((w[i] & 0x7fffu) != 0u && !(w[i] & 0x8000u) ? 1u : 0u) << (cb * 4 + r);
      mask |= (((w[i] >> 16) & 0x7fffu) != 0u && !(w[i] & 0x80000000u) ? 1u : 0u) << (cb * 4 + r + 1);
    }
  }
}
// Whether the value of T-order fragments hf at accumulator position
// (cb, r) is positive: bf16 bits with the sign clear and a nonzero
// magnitude, the test rt_relu_frags makes for its mask bit cb * 4 + r.
template <int NKH>
__device__ __forceinline__ bool rt_relu_on(const uint4 (&hf)[NKH], int cb, int r) {
  const uint4 f = hf[cb / 2];
  const int i = 2 * (cb % 2) + r / 2;
  const uint32_t w = i == 0 ? f.x : i == 1 ? f.y : i == 2 ? f.z : f.w;
  return (int32_t)(r % 2 ? (w & 0xffff0000u) : (w << 16)) > 0;
}
template <int NKH>
__device__ __forceinline__ void rt_load_relu(const uint16_t* __restrict__ hp, int q, uint4 (&hf)[NKH],
                                             uint32_t& mask) {
  uint4 raw[NKH];
#pragma unroll
  for (int kg = 0; kg < NKH; ++kg) raw[kg] = *reinterpret_cast<const uint4*>(hp + kg * 32 + q * 8);
  rt_relu_frags<NKH>(raw, hf, mask);
}

template <int NKH>
__device__ __forceinline__ void rt_store_frags(uint16_t* __restrict__ row, int q, const uint4 (&f)[NKH], bool ok) {
  uint4 p[NKH];
#pragma unroll
  for (int kg = 0; kg < NKH; ++kg) p[kg] = rt_to_plain(f[kg]);
  if (ok) {
#pragma unroll
    for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(row + kg * 32 + q * 8) = p[kg];
  }
}

// Sum over the four 16-lane groups; every lane gets the same bits.
__device__ __forceinline__ float rt_sum4(float x) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float s = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto p2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
  return __uint_as_float(p2[0]) + __uint_as_float(p2[1]);
}

// Per-lane partial over an accumulator tile's values, four chains.
template <int NB>
__device__ __forceinline__ float rt_lane_sum(const float (&v)[NB][4]) {
  float t[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    t[r] = v[0][r];
#pragma unroll
    for (int cb = 1; cb < NB; ++cb) t[r] += v[cb][r];
  }
  return (t[0] + t[1]) + (t[2] + t[3]);
}

// One reduce-scatter step within a 16-lane group: v[0, N) -> v[0, N / 2);
// the lane keeps the half that `hi` selects, summed with the DPP partner's
// copy of it (the partner keeps the other half).  Both halves' sums are
// formed, each one add with the partner's value read through DPP (every
// lane of these patterns has a partner in its row), and one is selected:
// three instructions per pair instead of two selects, a move and an add.
template <int N, int CTRL>
__device__ __forceinline__ void rt_halve(float* v, bool hi) {
  // no contraction with a product that formed v: both partners must add the
  // same two rounded values
#pragma clang fp contract(off)
#pragma unroll
  for (int k = 0; k < N / 2; ++k) {
    const float lo = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v[k]), CTRL, 0xf, 0xf, true)) + v[k];
    const float up =
        __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v[k + N / 2]), CTRL, 0xf, 0xf, true)) + v[k + N / 2];
    v[k] = hi ? up : lo;
  }
}

// Column totals over a tile's 16 rows.  In: v[NV] per lane (index 4 cb + r of
// the accumulator order).  Out: lane e's v[t], t < NV / 16, is the total of
// index e * NV / 16 + t.  Partners: row mirror (e ^ 15), half-row mirror
// (e ^ 7), then e ^ 3 and e ^ 1 within quads.
template <int NV>
__device__ __forceinline__ void rt_col_totals(float (&v)[NV], int e) {
  static_assert(NV >= 16, "at least one total per lane");
  rt_halve<NV, 0x140>(v, e & 8);
  rt_halve<NV / 2, 0x141>(v, e & 4);
  rt_halve<NV / 4, 0x1B>(v, e & 2);
  rt_halve<NV / 8, 0xB1>(v, e & 1);
}

// 4 consecutive floats of a plain-order row at column 16 cb + 4 q.
__device__ __forceinline__ float4 rt_ld4(const float* __restrict__ p, int cb, int q) {
  return *reinterpret_cast<const float4*>(p + cb * 16 + q * 4);
}

// z_1 of a tile in T order: W_e e (MFMA) + P_s[s] + P_r[r], added in that
// order, with b_1 inside P_r (the forward and the recompute in the backward
// share it).
template <int L>
__device__ __forceinline__ void rt_first_layer(const uint4 (&ef)[L / 32], const uint4* W1e, const RsMeta& mt, bool ok,
                                               const float* __restrict__ proj, floatx4 (&z)[L / 16], int lane) {
  constexpr int NB = L / 16;
  const int q = lane >> 4;
  // rows past the tile's end gather node 0 (their results are never used)
  const float* sp = proj + (int64_t)(ok ? mt.s : 0) * (2 * L);
  const float* rp = proj + (int64_t)(ok ? mt.r : 0) * (2 * L) + L;
  float4 ps[NB], pr[NB];
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) {
    ps[cb] = rt_ld4(sp, cb, q);
    pr[cb] = rt_ld4(rp, cb, q);
  }
  // the gathers issue before the products, which then hide their latency
  __builtin_amdgcn_sched_barrier(0);
  rt_gemm<NB, L / 32>(W1e, ef, z, lane);
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) {
    z[cb][0] = (z[cb][0] + ps[cb].x) + pr[cb].x;
    z[cb][1] = (z[cb][1] + ps[cb].y) + pr[cb].y;
    z[cb][2] = (z[cb][2] + ps[cb].z) + pr[cb].z;
    z[cb][3] = (z[cb][3] + ps[cb].w) + pr[cb].w;
  }
}

// Copies n floats into LDS (all threads of the workgroup).
__device__ __forceinline__ void rt_copy_vec(float* dst, const float* __restrict__ src, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src[i];
}

// Accumulator tile -> bf16 scratch (row order, swizzled) -> A fragments.
template <int L>
__device__ __forceinline__ void rs_to_frags(const float (&v)[L / 16][4], uint16_t* scr, uint4 (&f)[L / 32], int lane) {
  constexpr int NB = L / 16;
#pragma unroll
  for (int cb = 0; cb < NB; ++cb)
#pragma unroll
    for (int r = 0; r < 4; ++r) scr[rs_sw16<L>((lane >> 4) * 4 + r, cb * 16 + (lane & 15))] = f2bf(v[cb][r]);
#pragma unroll
  for (int kg = 0; kg < L / 32; ++kg)
    f[kg] = *reinterpret_cast<const uint4*>(scr + rs_sw16<L>(lane & 15, kg * 32 + (lane >> 4) * 8));
}

// n rows of a bf16 scratch tile -> consecutive global rows at dst.
template <int L>
__device__ __forceinline__ void rs_store_rows(uint16_t* __restrict__ dst, const uint16_t* scr, int n, int lane) {
  constexpr int CPR = L / 8;
  for (int i = lane; i < 16 * CPR; i += 64) {
    const int row = i / CPR, c = (i % CPR) * 8;
    if (row < n) *reinterpret_cast<uint4*>(dst + (int64_t)row * L + c) = *reinterpret_cast<const uint4*>(scr + rs_sw16<L>(row, c));
  }
}

// Per-lane partials of the lane's four rows -> row totals over the 16 lanes
// of the row group (butterfly; every lane of the group gets the same bits).
__device__ __forceinline__ void rs_butterfly(float (&t)[4]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float x = t[r];
    x += __shfl_xor(x, 1, 64);
    x += __shfl_xor(x, 2, 64);
    x += __shfl_xor(x, 4, 64);
    x += __shfl_xor(x, 8, 64);
    t[r] = x;
  }
}

// Row totals of an accumulator tile over all L columns.
template <int NB>
__device__ __forceinline__ void rs_row_totals(const float (&v)[NB][4], float (&t)[4]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float x = 0.f;
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) x += v[cb][r];
    t[r] = x;
  }
  rs_butterfly(t);
}

template <int L, int D>
struct RsFwdLay {
  static constexpr int NKH = L / 32, NB = L / 16;
  static constexpr int W = NB * NKH * 64 * 16;         // bytes of one L x L packed layer
  static constexpr int SCR = 16 * 64 * 4;              // per-wave scratch: 16 rows x 64 fp32 columns
  // vectors: last bias, gamma, beta[, hidden bias]
  static constexpr int OFF_W1 = 0, OFF_WH = W, OFF_WL = (D - 1) * W, OFF_VEC = D * W;
  static constexpr int NVEC = (D == 3 ? 4 : 3) * L;
  static constexpr int OFF_SCR = OFF_VEC + NVEC * 4;
  // 12 waves per workgroup (at most 168 registers each: a tile's gathers are
  // all in flight before its first product)
  static constexpr int NWV = 12;
  static constexpr int NTH = 64 * NWV;
  static constexpr int END = OFF_SCR + NWV * SCR;
  static_assert(END <= 160 * 1024, "LDS");
};

// Forward of one block's edge half (T form); P = node projections of the
// block input.
template <int L, int D>
__global__ __launch_bounds__((RsFwdLay<L, D>::NTH)) void edge_fwd_rs_kernel(EdgeFwdArgs a) {
  using Lay = RsFwdLay<L, D>;
  constexpr int NKH = Lay::NKH, NB = Lay::NB;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* W1 = reinterpret_cast<uint4*>(lds + Lay::OFF_W1);
  uint4* WH = reinterpret_cast<uint4*>(lds + Lay::OFF_WH);
  uint4* WL = reinterpret_cast<uint4*>(lds + Lay::OFF_WL);
  float* vbl = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // last bias
  float* vg = vbl + L;                                          // gamma
  float* vbt = vbl + 2 * L;                                     // beta
  float* vbh = vbl + 3 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  float* scr32 = reinterpret_cast<float*>(lds + Lay::OFF_SCR + wave * Lay::SCR);
  rs_copy_frags(W1, a.mlp.lin[0].wf, NB, NKH, 3 * NKH, 0);  // B operand read from memory rows
  if constexpr (D == 3) rt_copy_frags(WH, a.mlp.lin[1].wf, NB, NKH, NKH, 0);
  rt_copy_frags(WL, a.mlp.lin[D - 1].wf, NB, NKH, NKH, 0);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  rt_copy_vec(vbt, a.mlp.beta, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  __syncthreads();
  int64_t r0, r1;
  rs_range(a.row_ptr, 0, a.n_owned, r0, r1);
  rs_zero_empty(a.row_ptr, r0, r1, a.agg, L);
  const int64_t E0 = rs_uniform(a.row_ptr[r0]), E1 = rs_uniform(a.row_ptr[r1]);  // wave-uniform
  const uint16_t* Ein = reinterpret_cast<const uint16_t*>(a.Ein);
  uint16_t* Eout = reinterpret_cast<uint16_t*>(a.Eout);
  float run[(L + 63) / 64] = {};  // running receiver sums, columns lane + 64 j
  // the next tile's metadata is loaded when a tile starts and turned into
  // its mask before the tile's first store, so that the loop's head waits on
  // no store of the tile before
  RsMeta mt_next = rt_meta_make(rt_meta_load(a.erecv, a.send, E0, E1));
  for (int64_t sb = E0; sb < E1; sb += 16) {
    // an opaque copy of the lane index, so that the lane-dependent addresses
    // are recomputed per tile instead of being hoisted into registers
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int n = (int)(E1 - sb < 16 ? E1 - sb : 16);
    const bool ok = e < n;
    const RsMeta mt = mt_next;
    const RsMetaRaw nxt = rt_meta_load(a.erecv, a.send, sb + 16, E1);
    // rows past the tile's end repeat row 0 (their results are never stored)
    const int64_t er = sb + (ok ? e : 0);
    const uint16_t* erow = Ein + er * L;
    uint4 ef[NKH];
#pragma unroll
    for (int kg = 0; kg < NKH; ++kg) ef[kg] = *reinterpret_cast<const uint4*>(erow + kg * 32 + q * 8);
    floatx4 z[NB];
    rt_first_layer<L>(ef, W1, mt, ok, a.proj, z, ln);
    float h[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) h[cb][r] = z[cb][r] > 0.f ? z[cb][r] : 0.f;
    uint4 hf[NKH];
    rt_frags<NB>(h, hf);
    mt_next = rt_meta_make(nxt);
    if (a.hid_out) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid_out) + (sb + e) * L, q, hf, ok);
    if constexpr (D == 3) {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(WH, hf, acc, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 bv = rt_ld4(vbh, cb, q);
        const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v = acc[cb][r] + b4[r];
          h[cb][r] = v > 0.f ? v : 0.f;
        }
      }
      rt_frags<NB>(h, hf);
    }
    floatx4 acc[NB];
    rt_gemm<NB, NKH>(WL, hf, acc, ln);
    float y[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 bv = rt_ld4(vbl, cb, q);
      y[cb][0] = acc[cb][0] + bv.x;
      y[cb][1] = acc[cb][1] + bv.y;
      y[cb][2] = acc[cb][2] + bv.z;
      y[cb][3] = acc[cb][3] + bv.w;
    }
    // e^k in T order (4 columns per block) for the residual
    uint2 ev[NB];
#pragma unroll
    for (int kg = 0; kg < NKH; ++kg) {
      const uint4 t = rt_from_plain(ef[kg]);
      ev[2 * kg] = make_uint2(t.x, t.y);
      ev[2 * kg + 1] = make_uint2(t.z, t.w);
    }
    // LayerNorm: two-pass statistics of row e, then gamma * xhat + beta
    const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
    float dv[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float d = y[cb][r] - mu;
        dv[cb][r] = d * d;
      }
    const float rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
    // y becomes m
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 g = rt_ld4(vg, cb, q), bt = rt_ld4(vbt, cb, q);
      y[cb][0] = g.x * ((y[cb][0] - mu) * rs) + bt.x;
      y[cb][1] = g.y * ((y[cb][1] - mu) * rs) + bt.y;
      y[cb][2] = g.z * ((y[cb][2] - mu) * rs) + bt.z;
      y[cb][3] = g.w * ((y[cb][3] - mu) * rs) + bt.w;
      // e^{k+1} = e^k + m
      const uint2 w = ev[cb];
      ev[cb] = make_uint2(bf_pack(__uint_as_float(w.x << 16) + y[cb][0], __uint_as_float(w.x & 0xffff0000u) + y[cb][1]),
                          bf_pack(__uint_as_float(w.y << 16) + y[cb][2], __uint_as_float(w.y & 0xffff0000u) + y[cb][3]));
    }
    if (Eout) {
      uint4 o[NKH];
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg)
        o[kg] = rt_to_plain(make_uint4(ev[2 * kg].x, ev[2 * kg].y, ev[2 * kg + 1].x, ev[2 * kg + 1].y));
      if (ok) {
        uint16_t* orow = Eout + (sb + e) * L;
#pragma unroll
        for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(orow + kg * 32 + q * 8) = o[kg];
      }
    }
    // ordered receiver sums, 64 columns at a time through the wave's scratch
    // tile; a segment's total goes out at its last row
#pragma unroll
    for (int j = 0; j < (L + 63) / 64; ++j) {
      const int c = ln + 64 * j;
#pragma unroll
      for (int cb = 4 * j; cb < 4 * j + 4 && cb < NB; ++cb)
        *reinterpret_cast<float4*>(scr32 + rs_sw32<64>(e, (cb - 4 * j) * 16 + q * 4)) =
            make_float4(y[cb][0], y[cb][1], y[cb][2], y[cb][3]);
      float x[16];
#pragma unroll
      for (int row = 0; row < 16; ++row) x[row] = scr32[rs_sw32<64>(row, ln)];
#pragma unroll
      for (int row = 0; row < 16; ++row) {
        if (row < n) {
          run[j] += x[row];
          if ((mt.last >> row) & 1ull) {
            a.agg[(int64_t)__builtin_amdgcn_readlane(mt.r, row) * L + c] = run[j];
            run[j] = 0.f;
          }
        }
      }
    }
  }
}

template <int L, int D>
struct RsBwdLay {
  static constexpr int NKH = L / 32, NB = L / 16;
  static constexpr int W = NB * NKH * 64 * 16;
  static constexpr int SCR = 16 * 64 * 2;              // per-wave scratch: 16 rows x 64 bf16 columns
  // W_e (fwd), [W_h (fwd)], W_last (fwd), W_last (bwd), [W_h (bwd)], W_e (bwd)
  static constexpr int NW = D == 3 ? 6 : 4;
  static constexpr int OFF_VEC = NW * W;               // last bias, gamma[, hidden bias]
  static constexpr int OFF_SCR = OFF_VEC + (D == 3 ? 3 : 2) * L * 4;
  static constexpr int END = OFF_SCR + RS_NWV * SCR;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NVEC = (D + 2) * L;             // bias / gamma / beta partials per wave
  static_assert(RS_NWV * NVEC * 4 <= OFF_SCR, "partials reuse the weight area");
};

// Backward of one block's edge half (T form) with the tile's forward
// recomputed: dz_0 receiver sums over the consumed dagg rows, de^k, the
// stored gradients and activations, per-workgroup bias / LayerNorm partials.
// STASH: h_1 comes from the forward (a.hid_in, bf16, the block's edges in
// order) instead of W_e e + P_s + P_r, and is not stored again.
template <int L, int D, bool STASH>
__global__ __launch_bounds__(RS_NTH) void edge_bwd_rs_kernel(EdgeBwdArgs a) {
  using Lay = RsBwdLay<L, D>;
  constexpr int NKH = Lay::NKH, NB = Lay::NB, W = Lay::W;
  constexpr int NV = 4 * NB, NR = NV / 16;  // accumulator values per lane; column totals kept per lane
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* W1f = reinterpret_cast<uint4*>(lds);
  uint4* WHf = reinterpret_cast<uint4*>(lds + W);
  uint4* WLf = reinterpret_cast<uint4*>(lds + (D - 1) * W);
  uint4* WLb = reinterpret_cast<uint4*>(lds + D * W);
  uint4* WHb = reinterpret_cast<uint4*>(lds + (D + 1) * W);
  uint4* W1b = reinterpret_cast<uint4*>(lds + (Lay::NW - 1) * W);
  float* vbl = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // last bias
  float* vg = vbl + L;                                          // gamma
  float* vbh = vbl + 2 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  uint16_t* scr = reinterpret_cast<uint16_t*>(lds + Lay::OFF_SCR + wave * Lay::SCR);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  rs_copy_frags(W1f, a.mlp.lin[0].wf, NB, NKH, 3 * NKH, 0);  // B operand read from memory rows
  if constexpr (D == 3) rt_copy_frags(WHf, a.mlp.lin[1].wf, NB, NKH, NKH, 0);
  rt_copy_frags(WLf, a.mlp.lin[D - 1].wf, NB, NKH, NKH, 0);
  rt_copy_frags(WLb, a.mlp.lin[D - 1].wb, NB, NKH, NKH, 0);
  if constexpr (D == 3) rt_copy_frags(WHb, a.mlp.lin[1].wb, NB, NKH, NKH, 0);
  rt_copy_frags(W1b, a.mlp.lin[0].wb, NB, NKH, NKH, 0);  // e block: the first NB column blocks
  __syncthreads();
  int64_t r0, r1;
  rs_range(a.row_ptr, a.r_lo, a.r_hi, r0, r1);
  rs_zero_empty(a.row_ptr, r0, r1, a.dagg, L);
  const int64_t E0 = rs_uniform(a.row_ptr[r0]), E1 = rs_uniform(a.row_ptr[r1]);  // wave-uniform
  const uint16_t* Ein = reinterpret_cast<const uint16_t*>(a.Ein);
  // column totals of the bias / LayerNorm gradients (rt_col_totals' share of
  // each lane): gamma, beta, last bias, hidden biases
  constexpr int NQ = 2 + D;
  float qacc[NQ][NR];
#pragma unroll
  for (int k = 0; k < NQ; ++k)
#pragma unroll
    for (int t = 0; t < NR; ++t) qacc[k][t] = 0.f;
  float run[(L + 63) / 64] = {};
  // the next tile's metadata is loaded when a tile starts and turned into
  // its mask before the tile's first store, so that the loop's head waits on
  // no store of the tile before
  RsMeta mt_next = rt_meta_make(rt_meta_load(a.erecv, a.send, E0, E1));
  for (int64_t sb = E0; sb < E1; sb += 16) {
    // an opaque copy of the lane index, so that the lane-dependent addresses
    // are recomputed per tile instead of being hoisted into registers
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int n = (int)(E1 - sb < 16 ? E1 - sb : 16);
    const bool ok = e < n;
    const RsMeta mt = mt_next;
    const RsMetaRaw nxt = rt_meta_load(a.erecv, a.send, sb + 16, E1);
    const int64_t srow = (sb - a.e_base + e) * L;  // row of the stored gradients / activations
    // rows past the tile's end repeat row 0 (dm = 0 there, so they add nothing)
    const int64_t er = sb + (ok ? e : 0);
    // the tile's streamed rows, issued together before any is used, so that
    // their latencies overlap: the stashed h_1 (or e^k), the receivers' dagg
    // rows and de^{k+1} (bf16, plain order).  The last block has no de^{k+1}:
    // its loads then re-read the tile's own h_1 (or e^k) rows (cache hits)
    // and are replaced by zeros where they are used, so no load waits on a
    // branch.
    uint4 xr[NKH], dnr[NKH];
    float4 g4[NB];
    {
      const uint16_t* xp = (STASH ? reinterpret_cast<const uint16_t*>(a.hid_in) : Ein) + er * L;
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) xr[kg] = *reinterpret_cast<const uint4*>(xp + kg * 32 + q * 8);
      const float* gp = a.dagg + (int64_t)(ok ? mt.r : 0) * L;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) g4[cb] = rt_ld4(gp, cb, q);
      const uint16_t* dp = a.de_next ? reinterpret_cast<const uint16_t*>(a.de_next) + er * L : xp;
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) dnr[kg] = *reinterpret_cast<const uint4*>(dp + kg * 32 + q * 8);
    }
    __builtin_amdgcn_sched_barrier(0);
    uint32_t mask[2] = {0u, 0u};  // ReLU derivative of the hidden layers, bit cb * 4 + r
    float h[NB][4];
    uint4 hf[NKH];
    // STASH: h_1's fragments; the ReLU derivative of the first layer is read
    // off their signs where it is applied (rt_relu_on), so no mask is built
    uint4 h1f[NKH];
    if constexpr (STASH) {
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {
        h1f[kg] = rt_from_plain(xr[kg]);
        hf[kg] = h1f[kg];
      }
    } else {
      const uint4(&ef)[NKH] = xr;
      floatx4 z[NB];
      rt_first_layer<L>(ef, W1f, mt, ok, a.proj, z, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool on = z[cb][r] > 0.f;
          mask[0] |= (on ? 1u : 0u) << (cb * 4 + r);
          h[cb][r] = on ? z[cb][r] : 0.f;
        }
      rt_frags<NB>(h, hf);
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[0]) + srow, q, hf, ok);
    }
    if constexpr (D == 3) {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(WHf, hf, acc, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 bv = rt_ld4(vbh, cb, q);
        const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v = acc[cb][r] + b4[r];
          const bool on = v > 0.f;
          mask[1] |= (on ? 1u : 0u) << (cb * 4 + r);
          h[cb][r] = on ? v : 0.f;
        }
      }
      rt_frags<NB>(h, hf);
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[1]) + srow, q, hf, ok);
    }
    float y[NB][4];
    {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(WLf, hf, acc, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 bv = rt_ld4(vbl, cb, q);
        y[cb][0] = acc[cb][0] + bv.x;
        y[cb][1] = acc[cb][1] + bv.y;
        y[cb][2] = acc[cb][2] + bv.z;
        y[cb][3] = acc[cb][3] + bv.w;
      }
    }
    // dm = dagg[receiver] + de^{k+1}
    float dm[NB][4];
    float4 d4[NB];  // de^{k+1}, kept for de^k
    {
      const bool has_de = a.de_next != nullptr;
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {  // plain order -> T order
        const uint4 t = rt_from_plain(has_de ? dnr[kg] : make_uint4(0u, 0u, 0u, 0u));
        d4[2 * kg] = make_float4(__uint_as_float(t.x << 16), __uint_as_float(t.x & 0xffff0000u),
                                 __uint_as_float(t.y << 16), __uint_as_float(t.y & 0xffff0000u));
        d4[2 * kg + 1] = make_float4(__uint_as_float(t.z << 16), __uint_as_float(t.z & 0xffff0000u),
                                     __uint_as_float(t.w << 16), __uint_as_float(t.w & 0xffff0000u));
      }
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        dm[cb][0] = ok ? g4[cb].x + d4[cb].x : 0.f;
        dm[cb][1] = ok ? g4[cb].y + d4[cb].y : 0.f;
        dm[cb][2] = ok ? g4[cb].z + d4[cb].z : 0.f;
        dm[cb][3] = ok ? g4[cb].w + d4[cb].w : 0.f;
      }
    }
    // LayerNorm (recomputed): y becomes xhat
    const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
    float rs;
    {
      float dv[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = y[cb][r] - mu;
          dv[cb][r] = d * d;
        }
      rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
    }
    // LayerNorm backward: dy = rstd (dm g - mean(dm g) - xhat mean(dm g xhat))
    float t1, t2;
    {
      float d1[NB][4], d2[NB][4], tg[NV], tb[NV];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 g4 = rt_ld4(vg, cb, q);
        const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          y[cb][r] = (y[cb][r] - mu) * rs;
          const float d = dm[cb][r] * g[r];
          d1[cb][r] = d;
          d2[cb][r] = d * y[cb][r];
          tg[cb * 4 + r] = dm[cb][r] * y[cb][r];
          tb[cb * 4 + r] = dm[cb][r];
        }
      }
      t1 = rt_sum4(rt_lane_sum<NB>(d1));
      t2 = rt_sum4(rt_lane_sum<NB>(d2));
      rt_col_totals<NV>(tg, e);
      rt_col_totals<NV>(tb, e);
#pragma unroll
      for (int t = 0; t < NR; ++t) {
        qacc[0][t] += tg[t];
        qacc[1][t] += tb[t];
      }
    }
    float v[NB][4];
    {
      float tl[NV];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 g4 = rt_ld4(vg, cb, q);
        const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = dm[cb][r] * g[r];
          v[cb][r] = rs * (d - t1 / L - y[cb][r] * (t2 / L));
          tl[cb * 4 + r] = v[cb][r];
        }
      }
      rt_col_totals<NV>(tl, e);
#pragma unroll
      for (int t = 0; t < NR; ++t) qacc[2][t] += tl[t];
    }
    uint4 gf[NKH];
    rt_frags<NB>(v, gf);
    mt_next = rt_meta_make(nxt);
    rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[D - 1]) + srow, q, gf, ok);
    // hidden layers: dz_{j-1} = (dz_j W_j) * [z_{j-1} > 0]
#pragma unroll
    for (int j = D - 1; j >= 1; --j) {
      floatx4 acc[NB];
      if (j == D - 1) {
        rt_gemm<NB, NKH>(WLb, gf, acc, ln);
      } else {
        if constexpr (D == 3) rt_gemm<NB, NKH>(WHb, gf, acc, ln);
      }
      float th[NV];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool on = (STASH && j == 1) ? rt_relu_on<NKH>(h1f, cb, r) : ((mask[j - 1] >> (cb * 4 + r)) & 1u);
          v[cb][r] = on ? acc[cb][r] : 0.f;
          th[cb * 4 + r] = v[cb][r];
        }
      rt_col_totals<NV>(th, e);
#pragma unroll
      for (int t = 0; t < NR; ++t) qacc[3 + (j - 1)][t] += th[t];
      rt_frags<NB>(v, gf);
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[j - 1]) + srow, q, gf, ok);
    }
    // edge-stream gradient: de^k = de^{k+1} + dz_0 W_1[:, e-block], summed
    // in fp32 and stored as bf16 (the gradient of the bf16 edge stream)
    {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(W1b, gf, acc, ln);
      uint4 o[NKH];
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {
        const floatx4 a0 = acc[2 * kg], a1 = acc[2 * kg + 1];
        const float4 d0 = d4[2 * kg], d1 = d4[2 * kg + 1];
        o[kg] = rt_to_plain(make_uint4(bf_pack(a0[0] + d0.x, a0[1] + d0.y), bf_pack(a0[2] + d0.z, a0[3] + d0.w),
                                       bf_pack(a1[0] + d1.x, a1[1] + d1.y), bf_pack(a1[2] + d1.z, a1[3] + d1.w)));
      }
      if (ok) {
        uint16_t* op = reinterpret_cast<uint16_t*>(a.de_out) + (sb + e) * L;
#pragma unroll
        for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(op + kg * 32 + q * 8) = o[kg];
      }
    }
    // receiver sums of dz_0 (bf16, as it fed the products), ascending edge
    // order, 64 columns at a time through the wave's scratch tile
#pragma unroll
    for (int j = 0; j < (L + 63) / 64; ++j) {
      const int c = ln + 64 * j;
#pragma unroll
      for (int kg = 2 * j; kg < 2 * j + 2 && kg < NKH; ++kg) {
        const int c0 = (kg - 2 * j) * 32 + q * 4;
        *reinterpret_cast<uint2*>(scr + rs_sw16<64>(e, c0)) = make_uint2(gf[kg].x, gf[kg].y);
        *reinterpret_cast<uint2*>(scr + rs_sw16<64>(e, c0 + 16)) = make_uint2(gf[kg].z, gf[kg].w);
      }
      float x[16];
#pragma unroll
      for (int row = 0; row < 16; ++row) x[row] = bf2f(scr[rs_sw16<64>(row, ln)]);
#pragma unroll
      for (int row = 0; row < 16; ++row) {
        if (row < n) {
          run[j] += x[row];
          if ((mt.last >> row) & 1ull) {
            a.dagg[(int64_t)__builtin_amdgcn_readlane(mt.r, row) * L + c] = run[j];
            run[j] = 0.f;
          }
        }
      }
    }
  }
  // column partials: lane (e, q)'s totals are columns 16 cb + 4 q + r for
  // index e * NR + t = 4 cb + r; then the waves in order through LDS (the
  // weight area is free now)
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  {
    float* rw = red + wave * Lay::NVEC;
#pragma unroll
    for (int t = 0; t < NR; ++t) {
      const int i = (lane & 15) * NR + t;
      const int col = (i >> 2) * 16 + (lane >> 4) * 4 + (i & 3);
#pragma unroll
      for (int h = 0; h < D - 1; ++h) rw[h * L + col] = qacc[3 + h][t];
      rw[(D - 1) * L + col] = qacc[2][t];
      rw[D * L + col] = qacc[0][t];
      rw[(D + 1) * L + col] = qacc[1][t];
    }
  }
  __syncthreads();
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  for (int i = threadIdx.x; i < Lay::NVEC; i += RS_NTH) {
    float t = 0.f;
    for (int w = 0; w < RS_NWV; ++w) t += red[w * Lay::NVEC + i];
    vp[i] = t;
  }
}

// P[n] = [W_s v_n | W_r v_n + b_1] for the local nodes (T form, plain
// column order): the sender and receiver blocks of the edge MLP's first
// Linear on the bf16 block input, fp32 sums.
template <int L>
__global__ __launch_bounds__(RS_NTH) void node_proj_kernel(const uint16_t* __restrict__ V16, int64_t n_local, Lin w1,
                                                           float* __restrict__ proj) {
  constexpr int NKH = L / 32, NB = L / 16;
  constexpr int W = NB * NKH * 64 * 16;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* WS = reinterpret_cast<uint4*>(lds);
  uint4* WR = reinterpret_cast<uint4*>(lds + W);
  rs_copy_frags(WS, w1.wf, NB, NKH, 3 * NKH, NKH);
  rs_copy_frags(WR, w1.wf, NB, NKH, 3 * NKH, 2 * NKH);
  __syncthreads();
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int64_t ntiles = (n_local + 15) / 16;
  for (int64_t t = (int64_t)blockIdx.x * RS_NWV + wave; t < ntiles; t += (int64_t)gridDim.x * RS_NWV) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t node = t * 16 + e;
    const bool ok = node < n_local;
    const int64_t src = ok ? node : t * 16;  // rows past the end repeat the tile's first row (not stored)
    uint4 vf[NKH];
#pragma unroll
    for (int kg = 0; kg < NKH; ++kg) vf[kg] = *reinterpret_cast<const uint4*>(V16 + src * L + kg * 32 + q * 8);
#pragma unroll
    for (int side = 0; side < 2; ++side) {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(side == 0 ? WS : WR, vf, acc, ln);
      if (side == 1) {  // the first Linear's bias rides with the receiver half
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 bv = rt_ld4(w1.b, cb, q);
          acc[cb][0] += bv.x;
          acc[cb][1] += bv.y;
          acc[cb][2] += bv.z;
          acc[cb][3] += bv.w;
        }
      }
      if (ok) {
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
          *reinterpret_cast<float4*>(proj + node * (2 * L) + side * L + cb * 16 + q * 4) =
              make_float4(acc[cb][0], acc[cb][1], acc[cb][2], acc[cb][3]);
      }
    }
  }
}

// acc[cb] = sum over k-groups of A[kg] x B[cb][kg] with the B fragments read
// from the packed weights in memory (a layer too large to keep in LDS).
template <int NB, int NKG>
__device__ __forceinline__ void rs_gemm_g(const uint4 (&A)[NKG], const uint4* __restrict__ Bg, floatx4 (&acc)[NB],
                                          int lane) {
  // an opaque zero offset keeps the fragment loads inside the caller's loop
  int z0 = 0;
  asm volatile("" : "+v"(z0));
  const uint4* B = Bg + z0;
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) acc[cb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kg = 0; kg < NKG; ++kg) {
    uint4 b[NB];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) b[cb] = B[(cb * NKG + kg) * 64 + lane];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) PBF16::mma(acc[cb], A[kg], b[cb]);
  }
}

// ------------------------------------ streamed-weight T-form kernels, l = 256 ---
// bf16, latent 256.  One l x l bf16 layer is 128 KB, so the per-edge layers
// cannot all sit in LDS as in the row-split kernels above.  Instead each
// layer's packed fragments are streamed through LDS in chunks of four
// 16-column blocks x every k-group (32 KB, double-buffered): the
// workgroup's waves step through the chunks together, one barrier per
// chunk, and each wave applies every chunk to its own tile of NS x 16 edges
// (T form as above: the fragments are the MFMA A operand, the tile the B
// operand, and one layer's accumulators rounded to bf16 are the next
// layer's B operand as they stand).  A thread loads its share of the chunk
// after next from L2 into registers before the current chunk's products and
// writes the next chunk's share to LDS, so the stream overlaps the MFMAs.
// A chunk of a layer covers column blocks 4c .. 4c + 3 over every k-group,
// so those output columns are complete after it: bias, projections and
// ReLU are applied chunk by chunk.  The sequence of chunks is the same for
// every tile (the block's weights), so the stream runs on across tiles.

constexpr int RW_L = 256;                          // latent width of these kernels
constexpr int RW_NB = RW_L / 16;                   // 16-column blocks of a layer
constexpr int RW_NKH = RW_L / 32;                  // k-groups of an l-wide input
constexpr int RW_CB = 4;                           // column blocks per chunk
constexpr int RW_NC = RW_NB / RW_CB;               // chunks per layer
constexpr int RW_CHUNK = RW_CB * RW_NKH * 64;      // uint4 per chunk (32 KB)

// One layer's fragments in the stream: packed [cb][src_nkg][64 lanes],
// k-groups kg0 .. kg0 + RW_NKH - 1 of each column block.
struct RwSrc {
  const uint4* frags;
  int src_nkg, kg0;
};

// A thread's share of one chunk, held in registers between its load from
// L2 and its copy to LDS.  PERM: k-slots permuted for a B operand in
// accumulator (T) order, as rt_copy_frags does; else plain (B from rows).
template <int NTH>
struct RwStage {
  // native vectors (a uint4 struct copy can leave the stage in scratch memory)
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 v[RW_CHUNK / NTH];
};
// Thread tid's byte offset within a chunk's k-group run: element i = tid +
// j NTH of the share is column block i / 512 and k-group (i / 64) % 8 of the
// chunk, so with 512 % NTH == 0 the k-group is (j NTH % 512) / 64 + tid / 64
// and the column block j NTH / 512: the thread-dependent part is tid / 64
// k-groups plus the lane's place in a fragment (PERM: the 8-byte half at
// k-slot order, as rt_copy_frags permutes them).
template <bool PERM>
__device__ __forceinline__ uint32_t rw_thread_off() {
  const int tid = threadIdx.x, ln = tid & 63, q = ln >> 4, cc = ln & 15;
  const uint32_t lane = PERM ? (uint32_t)((cc + 16 * (q >> 1)) * 2 + (q & 1)) * 8u : (uint32_t)ln * 16u;
  return (uint32_t)(tid >> 6) * 1024u + lane;
}

template <int NTH, bool PERM>
__device__ __forceinline__ void rw_load(RwStage<NTH>& s, const RwSrc src, int c, uint32_t vo) {
  static_assert(NTH % 64 == 0 && (RW_NKH * 64) % NTH == 0, "a share's k-groups stay within one column block");
  // the uniform part of the addresses, kept opaque so that it is formed at
  // every call (scalar arithmetic) instead of being hoisted out of the tile
  // loop as dozens of live pointers, one set per chunk position; vo is the
  // thread's part (rw_thread_off)
  uint32_t u = (uint32_t)(c * RW_CB * src.src_nkg + src.kg0) * 1024u;
  asm volatile("" : "+s"(u));
  const char* base = reinterpret_cast<const char*>(src.frags) + u;
#pragma unroll
  for (int j = 0; j < RW_CHUNK / NTH; ++j) {
    constexpr int SPAN = RW_NKH * 64;  // elements per column block
    const uint32_t f = (uint32_t)((j * NTH) / SPAN * src.src_nkg + ((j * NTH) % SPAN) / 64) * 1024u + vo;
    if constexpr (PERM) {
      const uint2 lo = *reinterpret_cast<const uint2*>(base + f);
      const uint2 hi = *reinterpret_cast<const uint2*>(base + f + 512u);
      s.v[j] = typename RwStage<NTH>::u32x4{lo.x, lo.y, hi.x, hi.y};
    } else {
      s.v[j] = *reinterpret_cast<const typename RwStage<NTH>::u32x4*>(base + f);
    }
  }
}
template <int NTH>
__device__ __forceinline__ void rw_store(const RwStage<NTH>& s, uint4* buf) {
#pragma unroll
  for (int j = 0; j < RW_CHUNK / NTH; ++j)
    *reinterpret_cast<typename RwStage<NTH>::u32x4*>(buf + (int)threadIdx.x + j * NTH) = s.v[j];
}

// acc[s][4 c + cbl] = sum over k-groups of the chunk's fragments (LDS) times
// X[s][kg], for the NS 16-edge sub-tiles of the wave.  The fragments of
// k-group kg + RW_PF are read while the products of k-group kg are issued,
// so the LDS latency hides behind RW_PF k-groups of products.
#ifndef RW_PF
#define RW_PF 2
#endif
template <int NS, bool ZERO = true>
__device__ __forceinline__ void rw_gemm(int C, const uint4* buf, const uint4 (&X)[NS][RW_NKH],
                                        floatx4 (&acc)[NS][RW_NB], int lane) {
  constexpr int PF = RW_PF;
  if constexpr (ZERO) {
#pragma unroll
    for (int cbl = 0; cbl < RW_CB; ++cbl)
#pragma unroll
      for (int s = 0; s < NS; ++s) acc[s][C * RW_CB + cbl] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  uint4 w[PF + 1][RW_CB];
#pragma unroll
  for (int kg = 0; kg < PF; ++kg)
#pragma unroll
    for (int cbl = 0; cbl < RW_CB; ++cbl) w[kg][cbl] = buf[(cbl * RW_NKH + kg) * 64 + lane];
#pragma unroll
  for (int kg = 0; kg < RW_NKH; ++kg) {
    if (kg + PF < RW_NKH) {
#pragma unroll
      for (int cbl = 0; cbl < RW_CB; ++cbl) w[(kg + PF) % (PF + 1)][cbl] = buf[(cbl * RW_NKH + kg + PF) * 64 + lane];
    }
#pragma unroll
    for (int cbl = 0; cbl < RW_CB; ++cbl)
#pragma unroll
      for (int s = 0; s < NS; ++s) PBF16::mma(acc[s][C * RW_CB + cbl], w[kg % (PF + 1)][cbl], X[s][kg]);
  }
}

// bf16 plain-order 16-byte chunk (8 columns) -> its T-order values: cb 2 kg
// gets .x/.y, cb 2 kg + 1 gets .z/.w (columns 4 q + r of each block).
__device__ __forceinline__ void rw_unpack(const uint4 p, float (&lo)[4], float (&hi)[4]) {
  const uint4 t = rt_from_plain(p);
  lo[0] = __uint_as_float(t.x << 16);
  lo[1] = __uint_as_float(t.x & 0xffff0000u);
  lo[2] = __uint_as_float(t.y << 16);
  lo[3] = __uint_as_float(t.y & 0xffff0000u);
  hi[0] = __uint_as_float(t.z << 16);
  hi[1] = __uint_as_float(t.z & 0xffff0000u);
  hi[2] = __uint_as_float(t.w << 16);
  hi[3] = __uint_as_float(t.w & 0xffff0000u);
}

// Largest tile count over the workgroup's waves (every wave must take part
// in every chunk step of the stream).
__device__ __forceinline__ int rw_max_tiles(int mine, int* slot) {
  const int wave = wave_id(), nwv = blockDim.x >> 6;
  if ((threadIdx.x & 63) == 0) slot[wave] = mine;
  __syncthreads();
  int t = 0;
  for (int w = 0; w < nwv; ++w) t = slot[w] > t ? slot[w] : t;
  return t;
}

template <int D, int NS, int NWV>
struct RwFwdLay {
  static constexpr int NTH = 64 * NWV;
  static constexpr int TE = 16 * NS;                       // edges per wave and tile
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_VEC = 2 * RW_CHUNK * 16;        // last bias, gamma, beta[, hidden bias]
  static constexpr int NVEC = (D == 3 ? 4 : 3) * RW_L;
  static constexpr int OFF_SCR = OFF_VEC + NVEC * 4;
  static constexpr int SCR = 16 * 64 * 4;                  // per wave: 16 rows x 64 fp32 columns
  static constexpr int OFF_SLOT = OFF_SCR + NWV * SCR;
  static constexpr int END = OFF_SLOT + 64;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NCH = D * RW_NC;                    // chunks per tile
  static_assert(NCH % 2 == 0, "the stream's buffer parity repeats every tile");
};

// Forward of one block's edge half (l = 256, bf16): z_1 = W_e e + P_s[s] +
// P_r[r] (P = node projections with b_1 in the receiver half), ReLU,
// [W_h, ReLU,] W_last, LayerNorm; e^{k+1} = e^k + m; agg = ordered receiver
// sums of m; optionally h_1 kept for the backward.
template <int D, int NS, int NWV>
__global__ __launch_bounds__(64 * NWV) __attribute__((amdgpu_waves_per_eu(NWV == 4 ? 1 : 2, NWV == 4 ? 1 : 2)))
void edge_fwd_rw_kernel(EdgeFwdArgs a) {
  using Lay = RwFwdLay<D, NS, NWV>;
  constexpr int NTH = Lay::NTH, NB = RW_NB, NKH = RW_NKH, L = RW_L, TE = Lay::TE;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  float* vbl = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // last bias
  float* vg = vbl + L;                                          // gamma
  float* vbt = vbl + 2 * L;                                     // beta
  float* vbh = vbl + 3 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  float* scr32 = reinterpret_cast<float*>(lds + Lay::OFF_SCR + wave * Lay::SCR);
  const RwSrc src[3] = {{a.mlp.lin[0].wf, 3 * NKH, 0}, {a.mlp.lin[1].wf, NKH, 0}, {a.mlp.lin[D - 1].wf, NKH, 0}};
  // stream position p (chunk p % NCH of a tile): layer p / RW_NC (0: first,
  // D - 1: last), chunk p % RW_NC; only the first layer's B operand is plain
  const uint32_t vo_plain = rw_thread_off<false>(), vo_perm = rw_thread_off<true>();
  auto load = [&](RwStage<NTH>& st, int p) {
    const int pp = p % Lay::NCH, j = pp / RW_NC, c = pp % RW_NC;
    if (j == 0) rw_load<NTH, false>(st, src[0], c, vo_plain);
    else rw_load<NTH, true>(st, src[j == D - 1 ? 2 : 1], c, vo_perm);
  };
  RwStage<NTH> stg;
  load(stg, 0);
  rw_store<NTH>(stg, buf);
  load(stg, 1);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  rt_copy_vec(vbt, a.mlp.beta, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  int64_t r0, r1;
  rs_range(a.row_ptr, 0, a.n_owned, r0, r1);
  rs_zero_empty(a.row_ptr, r0, r1, a.agg, L);
  // wave-uniform bounds, kept in scalar registers
  const int64_t E0 = rs_uniform(a.row_ptr[r0]), E1 = rs_uniform(a.row_ptr[r1]);
  const int ntile = rw_max_tiles((int)((E1 - E0 + TE - 1) / TE), reinterpret_cast<int*>(lds + Lay::OFF_SLOT));
  const uint16_t* Ein = reinterpret_cast<const uint16_t*>(a.Ein);
  uint16_t* Eout = reinterpret_cast<uint16_t*>(a.Eout);
  float run[L / 64] = {};  // running receiver sums, columns lane + 64 j
  // one step of the stream: the next chunk's share to LDS, the one after
  // into registers (the barrier ending the previous step freed that buffer)
  auto advance = [&](int p) {
    rw_store<NTH>(stg, buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg, p + 2);
  };
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t sb0 = E0 + (int64_t)t * TE;
    const bool active = sb0 < E1;  // wave-uniform
    RsMeta mt[NS];
    bool ok[NS];
    uint4 xf[NS][NKH];  // B operand: e^k rows, then h_1 (, h_2)
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int64_t sb = sb0 + 16 * s;
      ok[s] = active && sb + e < E1;
      mt[s] = rt_meta_make(rt_meta_load(a.erecv, a.send, active ? sb : E0, active ? E1 : E0));
      const uint16_t* erow = Ein + (ok[s] ? sb + e : E0) * L;
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg)
        xf[s][kg] = active ? *reinterpret_cast<const uint4*>(erow + kg * 32 + q * 8) : make_uint4(0, 0, 0, 0);
    }
    floatx4 acc[NS][NB];
    // first layer: W_e e + P_s[s] + P_r[r], ReLU
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      advance(c);
      float4 ps[NS][RW_CB], pr[NS][RW_CB];
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const float* sp = a.proj + (int64_t)(ok[s] ? mt[s].s : 0) * (2 * L);
        const float* rp = a.proj + (int64_t)(ok[s] ? mt[s].r : 0) * (2 * L) + L;
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          ps[s][cbl] = active ? rt_ld4(sp, c * RW_CB + cbl, q) : make_float4(0.f, 0.f, 0.f, 0.f);
          pr[s][cbl] = active ? rt_ld4(rp, c * RW_CB + cbl, q) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      if (active) rw_gemm<NS>(c, buf + (c & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          floatx4& z = acc[s][c * RW_CB + cbl];
          const float4 a4 = ps[s][cbl], b4 = pr[s][cbl];
          z[0] = fmaxf((z[0] + a4.x) + b4.x, 0.f);
          z[1] = fmaxf((z[1] + a4.y) + b4.y, 0.f);
          z[2] = fmaxf((z[2] + a4.z) + b4.z, 0.f);
          z[3] = fmaxf((z[3] + a4.w) + b4.w, 0.f);
        }
      __syncthreads();
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[s][cb][r];
      rt_frags<NB>(h, xf[s]);
      if (a.hid_out && active)
        rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid_out) + (sb0 + 16 * s + e) * L, q, xf[s], ok[s]);
    }
    if constexpr (D == 3) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(RW_NC + c);
        if (active) rw_gemm<NS>(c, buf + ((RW_NC + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int cbl = 0; cbl < RW_CB; ++cbl) {
            const float4 bv = rt_ld4(vbh, c * RW_CB + cbl, q);
            floatx4& z = acc[s][c * RW_CB + cbl];
            z[0] = fmaxf(z[0] + bv.x, 0.f);
            z[1] = fmaxf(z[1] + bv.y, 0.f);
            z[2] = fmaxf(z[2] + bv.z, 0.f);
            z[3] = fmaxf(z[3] + bv.w, 0.f);
          }
        __syncthreads();
      }
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        float h[NB][4];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) h[cb][r] = acc[s][cb][r];
        rt_frags<NB>(h, xf[s]);
      }
    }
    // last layer (+ bias)
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      constexpr int P0 = (D - 1) * RW_NC;
      advance(P0 + c);
      if (active) rw_gemm<NS>(c, buf + ((P0 + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const float4 bv = rt_ld4(vbl, c * RW_CB + cbl, q);
          floatx4& z = acc[s][c * RW_CB + cbl];
          z[0] += bv.x;
          z[1] += bv.y;
          z[2] += bv.z;
          z[3] += bv.w;
        }
      __syncthreads();
    }
    if (!active) continue;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int64_t sb = sb0 + 16 * s;
      const int n = (int)(E1 - sb < 16 ? (E1 - sb > 0 ? E1 - sb : 0) : 16);
      float y[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) y[cb][r] = acc[s][cb][r];
      // LayerNorm: two-pass statistics of row e, then gamma * xhat + beta
      const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
      float dv[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = y[cb][r] - mu;
          dv[cb][r] = d * d;
        }
      const float rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 g = rt_ld4(vg, cb, q), bt = rt_ld4(vbt, cb, q);
        y[cb][0] = g.x * ((y[cb][0] - mu) * rs) + bt.x;
        y[cb][1] = g.y * ((y[cb][1] - mu) * rs) + bt.y;
        y[cb][2] = g.z * ((y[cb][2] - mu) * rs) + bt.z;
        y[cb][3] = g.w * ((y[cb][3] - mu) * rs) + bt.w;
      }
      if (Eout) {
        // e^{k+1} = e^k + m (e^k read again, plain order -> T order)
        const uint16_t* erow = Ein + (ok[s] ? sb + e : E0) * L;
        uint4 o[NKH];
#pragma unroll
        for (int kg = 0; kg < NKH; ++kg) {
          float lo[4], hi[4];
          rw_unpack(*reinterpret_cast<const uint4*>(erow + kg * 32 + q * 8), lo, hi);
          const float* m0 = y[2 * kg];
          const float* m1 = y[2 * kg + 1];
          o[kg] = rt_to_plain(make_uint4(bf_pack(lo[0] + m0[0], lo[1] + m0[1]), bf_pack(lo[2] + m0[2], lo[3] + m0[3]),
                                         bf_pack(hi[0] + m1[0], hi[1] + m1[1]), bf_pack(hi[2] + m1[2], hi[3] + m1[3])));
        }
        if (ok[s]) {
          uint16_t* orow = Eout + (sb + e) * L;
#pragma unroll
          for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(orow + kg * 32 + q * 8) = o[kg];
        }
      }
      // ordered receiver sums, 64 columns at a time through the wave's
      // scratch tile; a segment's total goes out at its last row
#pragma unroll
      for (int j = 0; j < L / 64; ++j) {
        const int cc = ln + 64 * j;
#pragma unroll
        for (int cb = 4 * j; cb < 4 * j + 4; ++cb)
          *reinterpret_cast<float4*>(scr32 + rs_sw32<64>(e, (cb - 4 * j) * 16 + q * 4)) =
              make_float4(y[cb][0], y[cb][1], y[cb][2], y[cb][3]);
        float x[16];
#pragma unroll
        for (int row = 0; row < 16; ++row) x[row] = scr32[rs_sw32<64>(row, ln)];
#pragma unroll
        for (int row = 0; row < 16; ++row) {
          if (row < n) {
            run[j] += x[row];
            if ((mt[s].last >> row) & 1ull) {
              a.agg[(int64_t)__builtin_amdgcn_readlane(mt[s].r, row) * L + cc] = run[j];
              run[j] = 0.f;
            }
          }
        }
      }
    }
  }
}


template <int D, bool STASH, int NWV_>
struct RwBwdLay {
  static constexpr int NWV = NWV_, NTH = 64 * NWV;
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_VEC = 2 * RW_CHUNK * 16;        // last bias, gamma[, hidden bias]
  static constexpr int OFF_SCR = OFF_VEC + (D == 3 ? 3 : 2) * RW_L * 4;
  static constexpr int SCR = 16 * 64 * 2;                  // per wave: 16 rows x 64 bf16 columns
  static constexpr int OFF_SLOT = OFF_SCR + NWV * SCR;
  static constexpr int END = OFF_SLOT + 64;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NVEC = (D + 2) * RW_L;              // hidden biases, last bias, gamma, beta
  static_assert(NWV * NVEC * 4 <= OFF_VEC, "the partials reuse the chunk buffers");
  // forward layers streamed (the first only when it is recomputed), then
  // the backward products of layers D-1 .. 0
  static constexpr int NFL = STASH ? D - 1 : D;
  static constexpr int NCH = (NFL + D) * RW_NC;
  static_assert(NCH % 2 == 0, "the stream's buffer parity repeats every tile");
};

// A stored bf16 ReLU output row (plain order) as T-order B fragments, and
// its ReLU mask (bit 4 cb + r set where the value is positive).
__device__ __forceinline__ void rw_load_relu(const uint16_t* __restrict__ hp, int q, uint4 (&hf)[RW_NKH],
                                             uint64_t& mask) {
#pragma unroll
  for (int kg = 0; kg < RW_NKH; ++kg) {
    hf[kg] = rt_from_plain(*reinterpret_cast<const uint4*>(hp + kg * 32 + q * 8));
    const uint32_t w[4] = {hf[kg].x, hf[kg].y, hf[kg].z, hf[kg].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // dword i: block 2 kg + i / 2, rows r = 2 (i % 2) .. + 1
      const int cb = 2 * kg + i / 2, r = 2 * (i % 2);
      mask |= (uint64_t)((w[i] & 0x7fffu) != 0u && !(w[i] & 0x8000u)) << (cb * 4 + r);
      mask |= (uint64_t)(((w[i] >> 16) & 0x7fffu) != 0u && !(w[i] & 0x80000000u)) << (cb * 4 + r + 1);
    }
  }
}

// Backward of one block's edge half, l = 256, bf16, weights streamed as in
// edge_fwd_rw_kernel.  Per 16-edge tile of a wave's receiver-aligned range
// (within the launch's receiver chunk [r_lo, r_hi)): the forward's first
// layer (recomputed from e^k and the block's node projections, or read from
// the forward's h_1 when STASH), the later layers, LayerNorm; dm = dagg[r]
// + de^{k+1}; LayerNorm backward; each layer's output gradient (stored for
// the weight gradients, with the hidden activations) down to dz_0; de^k =
// de^{k+1} + dz_0 W_e (bf16, in place); the ordered receiver sums of dz_0
// overwrite the consumed dagg rows; bias / LayerNorm column partials per
// workgroup.
template <int D, bool STASH, int NWV>
__global__ __launch_bounds__(64 * NWV) __attribute__((amdgpu_waves_per_eu(NWV == 4 ? 1 : 2, NWV == 4 ? 1 : 2)))
void edge_bwd_rw_kernel(EdgeBwdArgs a) {
  using Lay = RwBwdLay<D, STASH, NWV>;
  constexpr int NTH = Lay::NTH, NB = RW_NB, NKH = RW_NKH, L = RW_L;
  constexpr int NV = 4 * NB, NR = NV / 16;  // accumulator values per lane; column totals kept per lane
  constexpr int NFL = Lay::NFL, NCH = Lay::NCH;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  float* vbl = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // last bias
  float* vg = vbl + L;                                          // gamma
  float* vbh = vbl + 2 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  uint16_t* scr = reinterpret_cast<uint16_t*>(lds + Lay::OFF_SCR + wave * Lay::SCR);
  // the stream: forward layers (first layer: e block of W_1, rows from memory;
  // the others from accumulators), then backward layers D-1 .. 0 (packed
  // for dY W; the first Linear's e block is its first 16 column blocks)
  const RwSrc fsrc[3] = {{a.mlp.lin[0].wf, 3 * NKH, 0}, {a.mlp.lin[1].wf, NKH, 0}, {a.mlp.lin[D - 1].wf, NKH, 0}};
  const RwSrc bsrc[3] = {{a.mlp.lin[0].wb, NKH, 0}, {a.mlp.lin[1].wb, NKH, 0}, {a.mlp.lin[D - 1].wb, NKH, 0}};
  const uint32_t vo_plain = rw_thread_off<false>(), vo_perm = rw_thread_off<true>();
  auto load = [&](RwStage<NTH>& st, int p) {
    const int pp = p % NCH, j = pp / RW_NC, c = pp % RW_NC;
    if (j < NFL) {
      const int layer = STASH ? j + 1 : j;  // forward layer
      if (layer == 0) rw_load<NTH, false>(st, fsrc[0], c, vo_plain);
      else rw_load<NTH, true>(st, fsrc[layer == D - 1 ? 2 : 1], c, vo_perm);
    } else {
      const int layer = D - 1 - (j - NFL);  // backward product of this layer
      rw_load<NTH, true>(st, bsrc[layer == 0 ? 0 : (layer == D - 1 ? 2 : 1)], c, vo_perm);
    }
  };
  RwStage<NTH> stg[2];  // chunks p + 1 and p + 2 in flight at step p
  load(stg[0], 0);
  rw_store<NTH>(stg[0], buf);
  load(stg[1], 1);
  load(stg[0], 2);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  int64_t r0, r1;
  rs_range(a.row_ptr, a.r_lo, a.r_hi, r0, r1);
  rs_zero_empty(a.row_ptr, r0, r1, a.dagg, L);
  const int64_t E0 = rs_uniform(a.row_ptr[r0]), E1 = rs_uniform(a.row_ptr[r1]);  // wave-uniform
  const int ntile = rw_max_tiles((int)((E1 - E0 + 15) / 16), reinterpret_cast<int*>(lds + Lay::OFF_SLOT));
  const uint16_t* Ein = reinterpret_cast<const uint16_t*>(a.Ein);
  // column totals of the bias / LayerNorm gradients (rt_col_totals' share of
  // each lane): gamma, beta, last bias, hidden biases
  constexpr int NQ = 2 + D;
  float qacc[NQ][NR];
#pragma unroll
  for (int k = 0; k < NQ; ++k)
#pragma unroll
    for (int t = 0; t < NR; ++t) qacc[k][t] = 0.f;
  float run[L / 64] = {};
  auto advance = [&](int p) {
    rw_store<NTH>(stg[(p + 1) & 1], buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg[(p + 1) & 1], p + 3);
  };
  // the next tile's metadata is loaded when a tile starts and made into its
  // mask before the tile's last stores, so that no tile's start waits on
  // the stores of the tile before (the memory counter is in order)
  RsMeta mt_next = rt_meta_make(rt_meta_load(a.erecv, a.send, E0, E1));
  // rows of the tile's own input, read in place of de^{k+1} by the last
  // block (which has none; the values are then replaced by zeros)
  const uint16_t* xin = STASH ? reinterpret_cast<const uint16_t*>(a.hid_in) : Ein;
  const bool has_de = a.de_next != nullptr;
  // all ones with de^{k+1}, zero without: the loaded bits are masked rather
  // than selected, so that the loads are not moved into a branch
  const uint32_t de_mask = has_de ? 0xffffffffu : 0u;
  auto de_bits = [&](const uint4 r) {
    return make_uint4(r.x & de_mask, r.y & de_mask, r.z & de_mask, r.w & de_mask);
  };
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t sb = E0 + (int64_t)t * 16;
    const bool active = sb < E1;  // wave-uniform
    const int n = active ? (int)(E1 - sb < 16 ? E1 - sb : 16) : 0;
    const bool ok = e < n;
    const RsMeta mt = mt_next;
    const bool active_next = sb + 16 < E1;
    const RsMetaRaw nxt = rt_meta_load(a.erecv, a.send, active_next ? sb + 16 : E0, active_next ? E1 : E0);
    const int64_t srow = (sb - a.e_base + e) * L;  // row of the stored gradients / activations
    // rows past the tile's end repeat the tile's first row (dm = 0 there)
    const int64_t er = active ? sb + (ok ? e : 0) : E0;
    uint64_t mask[2] = {0ull, 0ull};  // ReLU derivative of the hidden layers, bit 4 cb + r
    uint4 xf[1][NKH];                  // B operand (one 16-edge sub-tile)
    floatx4 acc[1][NB];
    int p = 0;                         // stream position within the tile
    if constexpr (STASH) {
      if (active) rw_load_relu(reinterpret_cast<const uint16_t*>(a.hid_in) + er * L, q, xf[0], mask[0]);
    } else {
      const RsMeta* mp = &mt;
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg)
        xf[0][kg] = active ? *reinterpret_cast<const uint4*>(Ein + er * L + kg * 32 + q * 8) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        const float* sp = a.proj + (int64_t)(ok ? mp->s : 0) * (2 * L);
        const float* rp = a.proj + (int64_t)(ok ? mp->r : 0) * (2 * L) + L;
        float4 ps[RW_CB], pr[RW_CB];
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          ps[cbl] = active ? rt_ld4(sp, c * RW_CB + cbl, q) : make_float4(0.f, 0.f, 0.f, 0.f);
          pr[cbl] = active ? rt_ld4(rp, c * RW_CB + cbl, q) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const int cb = c * RW_CB + cbl;
          floatx4& z = acc[0][cb];
          const float4 a4 = ps[cbl], b4 = pr[cbl];
          const float zz[4] = {(z[0] + a4.x) + b4.x, (z[1] + a4.y) + b4.y, (z[2] + a4.z) + b4.z,
                               (z[3] + a4.w) + b4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const bool on = zz[r] > 0.f;
            mask[0] |= (uint64_t)on << (cb * 4 + r);
            z[r] = on ? zz[r] : 0.f;
          }
        }
        __syncthreads();
      }
      p += RW_NC;
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[0]) + srow, q, xf[0], ok);
    }
    if constexpr (D == 3) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const int cb = c * RW_CB + cbl;
          const float4 bv = rt_ld4(vbh, cb, q);
          const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
          floatx4& z = acc[0][cb];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = z[r] + b4[r];
            const bool on = v > 0.f;
            mask[1] |= (uint64_t)on << (cb * 4 + r);
            z[r] = on ? v : 0.f;
          }
        }
        __syncthreads();
      }
      p += RW_NC;
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[1]) + srow, q, xf[0], ok);
    }
    // dm = dagg[receiver] + de^{k+1}, loaded before the last layer's
    // products so that the loads overlap them
    float dm[NB][4];
    {
      const float* gp = a.dagg + (int64_t)(ok ? mt.r : 0) * L;
      const uint16_t* dp = (has_de ? reinterpret_cast<const uint16_t*>(a.de_next) : xin) + er * L;
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {
        float lo[4] = {0.f, 0.f, 0.f, 0.f}, hi[4] = {0.f, 0.f, 0.f, 0.f};
        float4 g0 = make_float4(0.f, 0.f, 0.f, 0.f), g1 = g0;
        if (active) {
          const uint4 raw = *reinterpret_cast<const uint4*>(dp + kg * 32 + q * 8);
          rw_unpack(de_bits(raw), lo, hi);
          g0 = rt_ld4(gp, 2 * kg, q);
          g1 = rt_ld4(gp, 2 * kg + 1, q);
        }
        dm[2 * kg][0] = ok ? g0.x + lo[0] : 0.f;
        dm[2 * kg][1] = ok ? g0.y + lo[1] : 0.f;
        dm[2 * kg][2] = ok ? g0.z + lo[2] : 0.f;
        dm[2 * kg][3] = ok ? g0.w + lo[3] : 0.f;
        dm[2 * kg + 1][0] = ok ? g1.x + hi[0] : 0.f;
        dm[2 * kg + 1][1] = ok ? g1.y + hi[1] : 0.f;
        dm[2 * kg + 1][2] = ok ? g1.z + hi[2] : 0.f;
        dm[2 * kg + 1][3] = ok ? g1.w + hi[3] : 0.f;
      }
    }
    // last layer + bias: y
    {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const float4 bv = rt_ld4(vbl, c * RW_CB + cbl, q);
          floatx4& z = acc[0][c * RW_CB + cbl];
          z[0] += bv.x;
          z[1] += bv.y;
          z[2] += bv.z;
          z[3] += bv.w;
        }
        __syncthreads();
      }
      p += RW_NC;
    }
    // LayerNorm recomputed (y becomes xhat), then its backward
    float gv[NB][4];  // the gradient being propagated (fp32, accumulator order)
    if (active) {
      float y[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) y[cb][r] = acc[0][cb][r];
      const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
      float s2 = 0.f;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = y[cb][r] - mu;
          s2 += d * d;
        }
      const float rs = 1.0f / sqrtf(rt_sum4(s2) / L + a.eps);
      float t1 = 0.f, t2 = 0.f;
      {
        float tg[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 g4 = rt_ld4(vg, cb, q);
          const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            y[cb][r] = (y[cb][r] - mu) * rs;
            const float d = dm[cb][r] * g[r];
            t1 += d;
            t2 += d * y[cb][r];
            tg[cb * 4 + r] = dm[cb][r] * y[cb][r];
          }
        }
        t1 = rt_sum4(t1);
        t2 = rt_sum4(t2);
        rt_col_totals<NV>(tg, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[0][tt] += tg[tt];
      }
      {
        float tb[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) tb[cb * 4 + r] = dm[cb][r];
        rt_col_totals<NV>(tb, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[1][tt] += tb[tt];
      }
      {
        float tl[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 g4 = rt_ld4(vg, cb, q);
          const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[cb][r] = rs * (dm[cb][r] * g[r] - t1 / L - y[cb][r] * (t2 / L));
            tl[cb * 4 + r] = gv[cb][r];
          }
        }
        rt_col_totals<NV>(tl, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[2][tt] += tl[tt];
      }
    } else {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) gv[cb][r] = 0.f;
    }
    rt_frags<NB>(gv, xf[0]);
    if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[D - 1]) + srow, q, xf[0], ok);
    // hidden layers: dz_{j-1} = (dz_j W_j) * [z_{j-1} > 0]
#pragma unroll
    for (int j = D - 1; j >= 1; --j) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
        __syncthreads();
      }
      p += RW_NC;
      if (active) {
        float th[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[cb][r] = ((mask[j - 1] >> (cb * 4 + r)) & 1ull) ? acc[0][cb][r] : 0.f;
            th[cb * 4 + r] = gv[cb][r];
          }
        rt_col_totals<NV>(th, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[3 + (j - 1)][tt] += th[tt];
      }
      rt_frags<NB>(gv, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[j - 1]) + srow, q, xf[0], ok);
    }
    // edge-stream gradient: de^k = de^{k+1} + dz_0 W_1[:, e-block], bf16
    {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
        __syncthreads();
      }
    }
    if (!active) continue;
    mt_next = rt_meta_make(nxt);
    {
      const uint16_t* dp = (has_de ? reinterpret_cast<const uint16_t*>(a.de_next) : xin) + er * L;
      uint4 raw[NKH];
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) raw[kg] = *reinterpret_cast<const uint4*>(dp + kg * 32 + q * 8);
      uint4 o[NKH];
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {
        float lo[4] = {0.f, 0.f, 0.f, 0.f}, hi[4] = {0.f, 0.f, 0.f, 0.f};
        rw_unpack(de_bits(raw[kg]), lo, hi);
        const floatx4 a0 = acc[0][2 * kg], a1 = acc[0][2 * kg + 1];
        o[kg] = rt_to_plain(make_uint4(bf_pack(a0[0] + lo[0], a0[1] + lo[1]), bf_pack(a0[2] + lo[2], a0[3] + lo[3]),
                                       bf_pack(a1[0] + hi[0], a1[1] + hi[1]), bf_pack(a1[2] + hi[2], a1[3] + hi[3])));
      }
      if (ok) {
        uint16_t* op = reinterpret_cast<uint16_t*>(a.de_out) + (sb + e) * L;
#pragma unroll
        for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(op + kg * 32 + q * 8) = o[kg];
      }
    }
    // receiver sums of dz_0 (bf16, as it fed the products), ascending edge
    // order, 64 columns at a time through the wave's scratch tile
#pragma unroll
    for (int j = 0; j < L / 64; ++j) {
      const int cc = ln + 64 * j;
#pragma unroll
      for (int kg = 2 * j; kg < 2 * j + 2; ++kg) {
        const int c0 = (kg - 2 * j) * 32 + q * 4;
        *reinterpret_cast<uint2*>(scr + rs_sw16<64>(e, c0)) = make_uint2(xf[0][kg].x, xf[0][kg].y);
        *reinterpret_cast<uint2*>(scr + rs_sw16<64>(e, c0 + 16)) = make_uint2(xf[0][kg].z, xf[0][kg].w);
      }
      float x[16];
#pragma unroll
      for (int row = 0; row < 16; ++row) x[row] = bf2f(scr[rs_sw16<64>(row, ln)]);
#pragma unroll
      for (int row = 0; row < 16; ++row) {
        if (row < n) {
          run[j] += x[row];
          if ((mt.last >> row) & 1ull) {
            a.dagg[(int64_t)__builtin_amdgcn_readlane(mt.r, row) * L + cc] = run[j];
            run[j] = 0.f;
          }
        }
      }
    }
  }
  // column partials: lane (e, q)'s totals are columns 16 cb + 4 q + r for
  // index e * NR + t = 4 cb + r; then the waves in order through LDS (the
  // chunk buffers are free now)
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  {
    float* rw = red + wave * Lay::NVEC;
#pragma unroll
    for (int tt = 0; tt < NR; ++tt) {
      const int i = (lane & 15) * NR + tt;
      const int col = (i >> 2) * 16 + (lane >> 4) * 4 + (i & 3);
#pragma unroll
      for (int h = 0; h < D - 1; ++h) rw[h * L + col] = qacc[3 + h][tt];
      rw[(D - 1) * L + col] = qacc[2][tt];
      rw[D * L + col] = qacc[0][tt];
      rw[(D + 1) * L + col] = qacc[1][tt];
    }
  }
  __syncthreads();
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  for (int i = threadIdx.x; i < Lay::NVEC; i += NTH) {
    float tsum = 0.f;
    for (int w = 0; w < Lay::NWV; ++w) tsum += red[w * Lay::NVEC + i];
    vp[i] = tsum;
  }
}

// ------------------------------------------ l = 256 node half (bf16) ---
// The node MLP of a block at l = 256 in the streamed-weight form of the edge
// kernels (weights in 32 KB chunks through LDS, T-form products, one 16-row
// tile per wave and step, contiguous row ranges per wave).  Forward: z_1 =
// W_1 [v | agg] + b_1, the v and agg k-ranges of each column chunk streamed
// one after the other, then ReLU, [W_h, ReLU,] W_last + b, LayerNorm, v + m
// (fp32 and its bf16 copy); the first Linear's ReLU output h_1 is kept for the
// backward when hid_out is set (only that when out is null: the backward's
// recompute).  Backward (from that h_1): the later layers recomputed,
// LayerNorm backward, each layer's output gradient (stored for the weight
// gradients, with h_2) down to dz_0, then dv = dm + dz_0 W_1[:, v] and dagg =
// dz_0 W_1[:, agg] (fp32); bias / LayerNorm column partials per workgroup.

// Rows [r0, r1) of unit q of W (contiguous 16-row tiles).
__device__ __forceinline__ void rw_row_tiles(int64_t rows, int64_t q, int64_t W, int64_t& t0, int64_t& t1) {
  const int64_t T = (rows + 15) / 16;
  t0 = T * q / W;
  t1 = T * (q + 1) / W;
}

template <int D>
struct RwNodeFwdLay {
  static constexpr int NWV = 8, NTH = 64 * NWV;
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_VEC = 2 * RW_CHUNK * 16;        // b_1, last bias, gamma, beta[, hidden bias]
  static constexpr int NVEC = (D == 3 ? 5 : 4) * RW_L;
  static constexpr int END = OFF_VEC + NVEC * 4;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NCH0 = 2 * RW_NC;                   // first layer: v and agg halves per column chunk
  static constexpr int NCH = NCH0 + (D - 1) * RW_NC;
  static_assert(NCH % 2 == 0 && NCH0 % 2 == 0, "the stream's buffer parity repeats every tile");
};

template <int D>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void rows_rw_fwd_kernel(RowsFwdArgs a) {
  using Lay = RwNodeFwdLay<D>;
  constexpr int NTH = Lay::NTH, NB = RW_NB, NKH = RW_NKH, L = RW_L;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  float* vb1 = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // first bias
  float* vbl = vb1 + L;                                         // last bias
  float* vg = vb1 + 2 * L;                                      // gamma
  float* vbt = vb1 + 3 * L;                                     // beta
  float* vbh = vb1 + 4 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  // forward packing of W_1: 2 NKH k-groups per column block, v then agg
  const RwSrc src0[2] = {{a.mlp.lin[0].wf, 2 * NKH, 0}, {a.mlp.lin[0].wf, 2 * NKH, NKH}};
  const RwSrc src[2] = {{a.mlp.lin[1].wf, NKH, 0}, {a.mlp.lin[D - 1].wf, NKH, 0}};
  // the whole MLP, or only the first layer (out null)
  const int nch = a.out ? Lay::NCH : Lay::NCH0;
  const uint32_t vo_plain = rw_thread_off<false>(), vo_perm = rw_thread_off<true>();
  auto load = [&](RwStage<NTH>& st, int p) {
    const int pp = p % nch;
    if (pp < Lay::NCH0) rw_load<NTH, false>(st, src0[pp & 1], pp >> 1, vo_plain);
    else {
      const int j = (pp - Lay::NCH0) / RW_NC + 1, c = (pp - Lay::NCH0) % RW_NC;  // layer 1 .. D-1
      rw_load<NTH, true>(st, src[j == D - 1 ? 1 : 0], c, vo_perm);
    }
  };
  RwStage<NTH> stg;
  load(stg, 0);
  rw_store<NTH>(stg, buf);
  load(stg, 1);
  rt_copy_vec(vb1, a.mlp.lin[0].b, L);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  rt_copy_vec(vbt, a.mlp.beta, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  int64_t t0, t1;
  rw_row_tiles(a.rows, (int64_t)blockIdx.x * Lay::NWV + wave, (int64_t)gridDim.x * Lay::NWV, t0, t1);
  // every wave takes part in every chunk step: the largest range's count
  const int64_t T = (a.rows + 15) / 16, Wt = (int64_t)gridDim.x * Lay::NWV;
  const int ntile = (int)((T + Wt - 1) / Wt);
  __syncthreads();
  const uint16_t* V16 = reinterpret_cast<const uint16_t*>(a.in0_16);
  auto advance = [&](int p) {
    rw_store<NTH>(stg, buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg, p + 2);
  };
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t tile = t0 + t;
    const bool active = tile < t1;  // wave-uniform
    const int64_t row = tile * 16 + e;
    const bool ok = active && row < a.rows;
    const int64_t src_row = ok ? row : (active ? tile * 16 : 0);  // rows past the end repeat the tile's first
    // first-layer B operands: v (bf16 copy), agg (fp32 rounded to bf16)
    uint4 xv[1][NKH], xa[1][NKH];
#pragma unroll
    for (int kg = 0; kg < NKH; ++kg) {
      xv[0][kg] = active ? *reinterpret_cast<const uint4*>(V16 + src_row * L + kg * 32 + q * 8) : make_uint4(0, 0, 0, 0);
      float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
      if (active) {
        const float* ap = a.in1 + src_row * L + kg * 32 + q * 8;
        x0 = reinterpret_cast<const float4*>(ap)[0];
        x1 = reinterpret_cast<const float4*>(ap)[1];
      }
      xa[0][kg] = make_uint4(bf_pack(x0.x, x0.y), bf_pack(x0.z, x0.w), bf_pack(x1.x, x1.y), bf_pack(x1.z, x1.w));
    }
    floatx4 acc[1][NB];
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      advance(2 * c);
      if (active) rw_gemm<1>(c, buf, xv, acc, ln);
      __syncthreads();
      advance(2 * c + 1);
      if (active) rw_gemm<1, false>(c, buf + RW_CHUNK, xa, acc, ln);
#pragma unroll
      for (int cbl = 0; cbl < RW_CB; ++cbl) {
        const float4 bv = rt_ld4(vb1, c * RW_CB + cbl, q);
        floatx4& z = acc[0][c * RW_CB + cbl];
        z[0] = fmaxf(z[0] + bv.x, 0.f);
        z[1] = fmaxf(z[1] + bv.y, 0.f);
        z[2] = fmaxf(z[2] + bv.z, 0.f);
        z[3] = fmaxf(z[3] + bv.w, 0.f);
      }
      __syncthreads();
    }
    uint4 xf[1][NKH];
    {
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
      if (a.hid_out && active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid_out) + row * L, q, xf[0], ok);
    }
    if (!a.out) continue;  // only h_1 wanted (launch-uniform)
    int p = Lay::NCH0;
    if constexpr (D == 3) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const float4 bv = rt_ld4(vbh, c * RW_CB + cbl, q);
          floatx4& z = acc[0][c * RW_CB + cbl];
          z[0] = fmaxf(z[0] + bv.x, 0.f);
          z[1] = fmaxf(z[1] + bv.y, 0.f);
          z[2] = fmaxf(z[2] + bv.z, 0.f);
          z[3] = fmaxf(z[3] + bv.w, 0.f);
        }
        __syncthreads();
      }
      p += RW_NC;
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
    }
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      advance(p + c);
      if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
      for (int cbl = 0; cbl < RW_CB; ++cbl) {
        const float4 bv = rt_ld4(vbl, c * RW_CB + cbl, q);
        floatx4& z = acc[0][c * RW_CB + cbl];
        z[0] += bv.x;
        z[1] += bv.y;
        z[2] += bv.z;
        z[3] += bv.w;
      }
      __syncthreads();
    }
    if (!active) continue;
    float y[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) y[cb][r] = acc[0][cb][r];
    const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
    float dv[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float d = y[cb][r] - mu;
        dv[cb][r] = d * d;
      }
    const float rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
    // v + gamma * xhat + beta
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 g = rt_ld4(vg, cb, q), bt = rt_ld4(vbt, cb, q), v = rt_ld4(a.in0 + src_row * L, cb, q);
      y[cb][0] = (g.x * ((y[cb][0] - mu) * rs) + bt.x) + v.x;
      y[cb][1] = (g.y * ((y[cb][1] - mu) * rs) + bt.y) + v.y;
      y[cb][2] = (g.z * ((y[cb][2] - mu) * rs) + bt.z) + v.z;
      y[cb][3] = (g.w * ((y[cb][3] - mu) * rs) + bt.w) + v.w;
    }
    if (ok) {
      float* op = reinterpret_cast<float*>(a.out) + row * L;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
        *reinterpret_cast<float4*>(op + cb * 16 + q * 4) = make_float4(y[cb][0], y[cb][1], y[cb][2], y[cb][3]);
    }
    if (a.out16) {
      uint4 o[NKH];
      rt_frags<NB>(y, o);
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.out16) + row * L, q, o, ok);
    }
  }
}

template <int D>
struct RwNodeBwdLay {
  static constexpr int NWV = 4, NTH = 64 * NWV;
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_VEC = 2 * RW_CHUNK * 16;        // last bias, gamma[, hidden bias]
  static constexpr int END = OFF_VEC + (D == 3 ? 3 : 2) * RW_L * 4;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NVEC = (D + 2) * RW_L;              // biases, gamma, beta
  static_assert(NWV * NVEC * 4 <= OFF_VEC, "the partials reuse the chunk buffers");
  // forward layers 1 .. D-1, backward products of layers D-1 .. 1, then the
  // first Linear's v and agg column halves
  static constexpr int NCH = 2 * (D - 1) * RW_NC + 2 * RW_NC;
  static_assert(NCH % 2 == 0, "the stream's buffer parity repeats every tile");
};

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void rows_rw_bwd_kernel(RowsBwdArgs a) {
  using Lay = RwNodeBwdLay<D>;
  constexpr int NTH = Lay::NTH, NB = RW_NB, NKH = RW_NKH, L = RW_L, NCH = Lay::NCH;
  constexpr int NV = 4 * NB, NR = NV / 16;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  float* vbl = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // last bias
  float* vg = vbl + L;                                          // gamma
  float* vbh = vbl + 2 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  // backward packing of W_1: 2 x NB column blocks (v, then agg inputs) of NKH k-groups
  const RwSrc fsrc[2] = {{a.mlp.lin[1].wf, NKH, 0}, {a.mlp.lin[D - 1].wf, NKH, 0}};
  const RwSrc bsrc[2] = {{a.mlp.lin[1].wb, NKH, 0}, {a.mlp.lin[D - 1].wb, NKH, 0}};
  const RwSrc isrc[2] = {{a.mlp.lin[0].wb, NKH, 0}, {a.mlp.lin[0].wb + (size_t)NB * NKH * 64, NKH, 0}};
  const uint32_t vo_perm = rw_thread_off<true>();
  auto load = [&](RwStage<NTH>& st, int p) {
    const int pp = p % NCH, j = pp / RW_NC, c = pp % RW_NC;
    if (j < D - 1) rw_load<NTH, true>(st, fsrc[j == D - 2 ? 1 : 0], c, vo_perm);  // forward layer j + 1
    else if (j < 2 * (D - 1)) {
      const int layer = D - 1 - (j - (D - 1));                                 // backward product, D-1 .. 1
      rw_load<NTH, true>(st, bsrc[layer == D - 1 ? 1 : 0], c, vo_perm);
    } else {
      rw_load<NTH, true>(st, isrc[j - 2 * (D - 1)], c, vo_perm);               // dv, then dagg
    }
  };
  RwStage<NTH> stg[2];  // chunks p + 1 and p + 2 in flight at step p
  load(stg[0], 0);
  rw_store<NTH>(stg[0], buf);
  load(stg[1], 1);
  load(stg[0], 2);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  int64_t t0, t1;
  rw_row_tiles(a.rows, (int64_t)blockIdx.x * Lay::NWV + wave, (int64_t)gridDim.x * Lay::NWV, t0, t1);
  const int64_t T = (a.rows + 15) / 16, Wt = (int64_t)gridDim.x * Lay::NWV;
  const int ntile = (int)((T + Wt - 1) / Wt);
  __syncthreads();
  // column totals (rt_col_totals' share of each lane): gamma, beta, last
  // bias, hidden biases
  constexpr int NQ = 2 + D;
  float qacc[NQ][NR];
#pragma unroll
  for (int k = 0; k < NQ; ++k)
#pragma unroll
    for (int t = 0; t < NR; ++t) qacc[k][t] = 0.f;
  auto advance = [&](int p) {
    rw_store<NTH>(stg[(p + 1) & 1], buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg[(p + 1) & 1], p + 3);
  };
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t tile = t0 + t;
    const bool active = tile < t1;  // wave-uniform
    const int64_t row = tile * 16 + e;
    const bool ok = active && row < a.rows;
    const int64_t src_row = ok ? row : (active ? tile * 16 : 0);
    uint64_t mask[2] = {0ull, 0ull};  // ReLU derivative of the hidden layers, bit 4 cb + r
    uint4 xf[1][NKH];
    floatx4 acc[1][NB];
    int p = 0;
    if (active) rw_load_relu(reinterpret_cast<const uint16_t*>(a.hid_in) + src_row * L, q, xf[0], mask[0]);
    if constexpr (D == 3) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const int cb = c * RW_CB + cbl;
          const float4 bv = rt_ld4(vbh, cb, q);
          const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
          floatx4& z = acc[0][cb];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = z[r] + b4[r];
            const bool on = v > 0.f;
            mask[1] |= (uint64_t)on << (cb * 4 + r);
            z[r] = on ? v : 0.f;
          }
        }
        __syncthreads();
      }
      p += RW_NC;
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[1]) + row * L, q, xf[0], ok);
    }
    // dm (fp32), loaded before the last layer's products
    float dm[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      float4 d4 = make_float4(0.f, 0.f, 0.f, 0.f);
      if (active) d4 = rt_ld4(a.dm + src_row * L, cb, q);
      dm[cb][0] = ok ? d4.x : 0.f;
      dm[cb][1] = ok ? d4.y : 0.f;
      dm[cb][2] = ok ? d4.z : 0.f;
      dm[cb][3] = ok ? d4.w : 0.f;
    }
    // last layer + bias: y
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      advance(p + c);
      if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
      for (int cbl = 0; cbl < RW_CB; ++cbl) {
        const float4 bv = rt_ld4(vbl, c * RW_CB + cbl, q);
        floatx4& z = acc[0][c * RW_CB + cbl];
        z[0] += bv.x;
        z[1] += bv.y;
        z[2] += bv.z;
        z[3] += bv.w;
      }
      __syncthreads();
    }
    p += RW_NC;
    // LayerNorm recomputed (y becomes xhat), then its backward
    float gv[NB][4];
    if (active) {
      float y[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) y[cb][r] = acc[0][cb][r];
      const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
      float s2 = 0.f;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = y[cb][r] - mu;
          s2 += d * d;
        }
      const float rs = 1.0f / sqrtf(rt_sum4(s2) / L + a.eps);
      float t1s = 0.f, t2s = 0.f;
      {
        float tg[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 g4 = rt_ld4(vg, cb, q);
          const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            y[cb][r] = (y[cb][r] - mu) * rs;
            const float d = dm[cb][r] * g[r];
            t1s += d;
            t2s += d * y[cb][r];
            tg[cb * 4 + r] = dm[cb][r] * y[cb][r];
          }
        }
        t1s = rt_sum4(t1s);
        t2s = rt_sum4(t2s);
        rt_col_totals<NV>(tg, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[0][tt] += tg[tt];
      }
      {
        float tb[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) tb[cb * 4 + r] = dm[cb][r];
        rt_col_totals<NV>(tb, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[1][tt] += tb[tt];
      }
      {
        float tl[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 g4 = rt_ld4(vg, cb, q);
          const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[cb][r] = rs * (dm[cb][r] * g[r] - t1s / L - y[cb][r] * (t2s / L));
            tl[cb * 4 + r] = gv[cb][r];
          }
        }
        rt_col_totals<NV>(tl, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[2][tt] += tl[tt];
      }
    } else {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) gv[cb][r] = 0.f;
    }
    rt_frags<NB>(gv, xf[0]);
    if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[D - 1]) + row * L, q, xf[0], ok);
    // hidden layers: dz_{j-1} = (dz_j W_j) * [z_{j-1} > 0]
#pragma unroll
    for (int j = D - 1; j >= 1; --j) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
        __syncthreads();
      }
      p += RW_NC;
      if (active) {
        float th[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[cb][r] = ((mask[j - 1] >> (cb * 4 + r)) & 1ull) ? acc[0][cb][r] : 0.f;
            th[cb * 4 + r] = gv[cb][r];
          }
        rt_col_totals<NV>(th, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[3 + (j - 1)][tt] += th[tt];
      }
      rt_frags<NB>(gv, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[j - 1]) + row * L, q, xf[0], ok);
    }
    // input gradients: dv = dm + dz_0 W_1[:, v-block], dagg = dz_0 W_1[:, agg-block]
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
        __syncthreads();
      }
      p += RW_NC;
      if (ok) {
        float* op = (pass == 0 ? a.dx0 : a.dx1) + row * L;
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          floatx4 v = acc[0][cb];
          if (pass == 0) {
            v[0] += dm[cb][0];
            v[1] += dm[cb][1];
            v[2] += dm[cb][2];
            v[3] += dm[cb][3];
          }
          *reinterpret_cast<float4*>(op + cb * 16 + q * 4) = make_float4(v[0], v[1], v[2], v[3]);
        }
      }
    }
  }
  // column partials: lane (e, q)'s totals are columns 16 cb + 4 q + r for
  // index e * NR + t = 4 cb + r; then the waves in order through LDS (the
  // chunk buffers are free now)
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  {
    float* rw = red + wave * Lay::NVEC;
#pragma unroll
    for (int tt = 0; tt < NR; ++tt) {
      const int i = (lane & 15) * NR + tt;
      const int col = (i >> 2) * 16 + (lane >> 4) * 4 + (i & 3);
#pragma unroll
      for (int h = 0; h < D - 1; ++h) rw[h * L + col] = qacc[3 + h][tt];
      rw[(D - 1) * L + col] = qacc[2][tt];
      rw[D * L + col] = qacc[0][tt];
      rw[(D + 1) * L + col] = qacc[1][tt];
    }
  }
  __syncthreads();
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  for (int i = threadIdx.x; i < Lay::NVEC; i += NTH) {
    float tsum = 0.f;
    for (int w = 0; w < Lay::NWV; ++w) tsum += red[w * Lay::NVEC + i];
    vp[i] = tsum;
  }
}

// The edge encoder at l = 256 (bf16) in the same streamed-weight form: its
// first Linear (input fin <= 4 features, one k-group) stays in LDS for the
// whole launch, the later layers stream.  Forward: e^0 = LN(MLP(x)) (bf16
// rows).  Backward: the tile's forward recomputed from x, LayerNorm
// backward, each layer's output gradient (stored for the weight gradients,
// with h_1 and h_2) down to dz_0, whose product with x (the first Linear's
// weight gradient, 256 x fin) each wave accumulates itself: per tile dz_0 and
// x pass through a per-wave LDS scratch and lane l sums output rows 4 l ..
// 4 l + 3; bias / LayerNorm column partials per workgroup.
constexpr int RW_ENC_FIN = 4;

// The tile's first-Linear B operand from fin <= 4 fp32 features (lane group
// 0 holds k-slots 0 .. 7, the others zero), rounded to bf16.
__device__ __forceinline__ uint4 rw_enc_input(const float* __restrict__ x, int fin, int64_t row, int q, bool active) {
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (active && q == 0) {
#pragma unroll
    for (int j = 0; j < RW_ENC_FIN; ++j)
      if (j < fin) v[j] = x[row * fin + j];
  }
  return make_uint4(bf_pack(v[0], v[1]), bf_pack(v[2], v[3]), bf_pack(v[4], v[5]), bf_pack(v[6], v[7]));
}

// z_1 = W_1 x + b_1 over every column block, ReLU (mask bits when asked), as
// accumulators; W_1's NB fragments (one k-group) in LDS.
__device__ __forceinline__ void rw_enc_first(const uint4* W0, const float* vb1, const uint4 x, int lane,
                                             floatx4 (&acc)[1][RW_NB], uint64_t* mask) {
  const int q = lane >> 4;
#pragma unroll
  for (int cb = 0; cb < RW_NB; ++cb) {
    acc[0][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    PBF16::mma(acc[0][cb], W0[cb * 64 + lane], x);
    const float4 bv = rt_ld4(vb1, cb, q);
    const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v = acc[0][cb][r] + b4[r];
      const bool on = v > 0.f;
      if (mask) *mask |= (uint64_t)on << (cb * 4 + r);
      acc[0][cb][r] = on ? v : 0.f;
    }
  }
}

template <int D>
struct RwEncFwdLay {
  static constexpr int NWV = 8, NTH = 64 * NWV;
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_W0 = 2 * RW_CHUNK * 16;         // first Linear, NB fragments
  static constexpr int OFF_VEC = OFF_W0 + RW_NB * 64 * 16;  // b_1, last bias, gamma, beta[, hidden bias]
  static constexpr int END = OFF_VEC + (D == 3 ? 5 : 4) * RW_L * 4;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NCH = (D - 1) * RW_NC;
  static_assert(NCH % 2 == 0, "the stream's buffer parity repeats every tile");
};

template <int D>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void rows_rw_enc_fwd_kernel(RowsFwdArgs a) {
  using Lay = RwEncFwdLay<D>;
  constexpr int NTH = Lay::NTH, NB = RW_NB, NKH = RW_NKH, L = RW_L, NCH = Lay::NCH;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  uint4* W0 = reinterpret_cast<uint4*>(lds + Lay::OFF_W0);
  float* vb1 = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // first bias
  float* vbl = vb1 + L;                                         // last bias
  float* vg = vb1 + 2 * L;                                      // gamma
  float* vbt = vb1 + 3 * L;                                     // beta
  float* vbh = vb1 + 4 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const RwSrc src[2] = {{a.mlp.lin[1].wf, NKH, 0}, {a.mlp.lin[D - 1].wf, NKH, 0}};
  const uint32_t vo_perm = rw_thread_off<true>();
  auto load = [&](RwStage<NTH>& st, int p) {
    const int pp = p % NCH, j = pp / RW_NC + 1, c = pp % RW_NC;  // layer 1 .. D-1
    rw_load<NTH, true>(st, src[j == D - 1 ? 1 : 0], c, vo_perm);
  };
  RwStage<NTH> stg;
  load(stg, 0);
  rw_store<NTH>(stg, buf);
  load(stg, 1);
  rs_copy_frags(W0, a.mlp.lin[0].wf, NB, 1, a.mlp.lin[0].nkgf, 0);
  rt_copy_vec(vb1, a.mlp.lin[0].b, L);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  rt_copy_vec(vbt, a.mlp.beta, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  int64_t t0, t1;
  rw_row_tiles(a.rows, (int64_t)blockIdx.x * Lay::NWV + wave, (int64_t)gridDim.x * Lay::NWV, t0, t1);
  const int64_t T = (a.rows + 15) / 16, Wt = (int64_t)gridDim.x * Lay::NWV;
  const int ntile = (int)((T + Wt - 1) / Wt);
  __syncthreads();
  auto advance = [&](int p) {
    rw_store<NTH>(stg, buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg, p + 2);
  };
  uint16_t* out = reinterpret_cast<uint16_t*>(a.out);
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t tile = t0 + t;
    const bool active = tile < t1;  // wave-uniform
    const int64_t row = tile * 16 + e;
    const bool ok = active && row < a.rows;
    const int64_t src_row = ok ? row : (active ? tile * 16 : 0);
    floatx4 acc[1][NB];
    rw_enc_first(W0, vb1, rw_enc_input(a.in0, a.fin, src_row, q, active), ln, acc, nullptr);
    uint4 xf[1][NKH];
    {
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
    }
    int p = 0;
    if constexpr (D == 3) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const float4 bv = rt_ld4(vbh, c * RW_CB + cbl, q);
          floatx4& z = acc[0][c * RW_CB + cbl];
          z[0] = fmaxf(z[0] + bv.x, 0.f);
          z[1] = fmaxf(z[1] + bv.y, 0.f);
          z[2] = fmaxf(z[2] + bv.z, 0.f);
          z[3] = fmaxf(z[3] + bv.w, 0.f);
        }
        __syncthreads();
      }
      p += RW_NC;
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
    }
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      advance(p + c);
      if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
      for (int cbl = 0; cbl < RW_CB; ++cbl) {
        const float4 bv = rt_ld4(vbl, c * RW_CB + cbl, q);
        floatx4& z = acc[0][c * RW_CB + cbl];
        z[0] += bv.x;
        z[1] += bv.y;
        z[2] += bv.z;
        z[3] += bv.w;
      }
      __syncthreads();
    }
    if (!active) continue;
    float y[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) y[cb][r] = acc[0][cb][r];
    const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
    float dv[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float d = y[cb][r] - mu;
        dv[cb][r] = d * d;
      }
    const float rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 g = rt_ld4(vg, cb, q), bt = rt_ld4(vbt, cb, q);
      y[cb][0] = g.x * ((y[cb][0] - mu) * rs) + bt.x;
      y[cb][1] = g.y * ((y[cb][1] - mu) * rs) + bt.y;
      y[cb][2] = g.z * ((y[cb][2] - mu) * rs) + bt.z;
      y[cb][3] = g.w * ((y[cb][3] - mu) * rs) + bt.w;
    }
    uint4 o[NKH];
    rt_frags<NB>(y, o);
    rt_store_frags<NKH>(out + row * L, q, o, ok);
  }
}

template <int D>
struct RwEncBwdLay {
  static constexpr int NWV = 4, NTH = 64 * NWV;
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_W0 = 2 * RW_CHUNK * 16;         // first Linear, NB fragments
  static constexpr int OFF_VEC = OFF_W0 + RW_NB * 64 * 16;  // b_1, last bias, gamma[, hidden bias]
  static constexpr int OFF_SCR = OFF_VEC + (D == 3 ? 4 : 3) * RW_L * 4;
  // per wave: a tile's dz_0 (16 rows of l bf16, 8 columns of padding) and features
  static constexpr int DZS = RW_L + 8;
  static constexpr int SCR = 16 * DZS * 2 + 16 * RW_ENC_FIN * 2;
  static constexpr int END = OFF_SCR + NWV * SCR;
  static_assert(END <= 160 * 1024, "LDS");
  static constexpr int NVEC = (D + 2) * RW_L;              // biases, gamma, beta
  static_assert(NWV * NVEC * 4 <= OFF_W0, "the partials reuse the chunk buffers");
  // forward layers 1 .. D-1, then the backward products of layers D-1 .. 1
  static constexpr int NCH = 2 * (D - 1) * RW_NC;
  static_assert(NCH % 2 == 0, "the stream's buffer parity repeats every tile");
};

template <int D>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void rows_rw_enc_bwd_kernel(RowsBwdArgs a) {
  using Lay = RwEncBwdLay<D>;
  constexpr int NTH = Lay::NTH, NB = RW_NB, NKH = RW_NKH, L = RW_L, NCH = Lay::NCH;
  constexpr int NV = 4 * NB, NR = NV / 16, OPL = L / 64;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  uint4* W0 = reinterpret_cast<uint4*>(lds + Lay::OFF_W0);
  float* vb1 = reinterpret_cast<float*>(lds + Lay::OFF_VEC);  // first bias
  float* vbl = vb1 + L;                                         // last bias
  float* vg = vb1 + 2 * L;                                      // gamma
  float* vbh = vb1 + 3 * L;                                     // hidden bias (D = 3)
  const int wave = wave_id(), lane = threadIdx.x & 63;
  uint16_t* dzs = reinterpret_cast<uint16_t*>(lds + Lay::OFF_SCR + wave * Lay::SCR);
  uint16_t* xs = dzs + 16 * Lay::DZS;
  const RwSrc fsrc[2] = {{a.mlp.lin[1].wf, NKH, 0}, {a.mlp.lin[D - 1].wf, NKH, 0}};
  const RwSrc bsrc[2] = {{a.mlp.lin[1].wb, NKH, 0}, {a.mlp.lin[D - 1].wb, NKH, 0}};
  const uint32_t vo_perm = rw_thread_off<true>();
  auto load = [&](RwStage<NTH>& st, int p) {
    const int pp = p % NCH, j = pp / RW_NC, c = pp % RW_NC;
    if (j < D - 1) rw_load<NTH, true>(st, fsrc[j == D - 2 ? 1 : 0], c, vo_perm);  // forward layer j + 1
    else {
      const int layer = D - 1 - (j - (D - 1));                                 // backward product, D-1 .. 1
      rw_load<NTH, true>(st, bsrc[layer == D - 1 ? 1 : 0], c, vo_perm);
    }
  };
  RwStage<NTH> stg[2];  // chunks p + 1 and p + 2 in flight at step p
  load(stg[0], 0);
  rw_store<NTH>(stg[0], buf);
  load(stg[1], 1);
  load(stg[0], 2);
  rs_copy_frags(W0, a.mlp.lin[0].wf, NB, 1, a.mlp.lin[0].nkgf, 0);
  rt_copy_vec(vb1, a.mlp.lin[0].b, L);
  rt_copy_vec(vbl, a.mlp.lin[D - 1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  if constexpr (D == 3) rt_copy_vec(vbh, a.mlp.lin[1].b, L);
  int64_t t0, t1;
  rw_row_tiles(a.rows, (int64_t)blockIdx.x * Lay::NWV + wave, (int64_t)gridDim.x * Lay::NWV, t0, t1);
  const int64_t T = (a.rows + 15) / 16, Wt = (int64_t)gridDim.x * Lay::NWV;
  const int ntile = (int)((T + Wt - 1) / Wt);
  __syncthreads();
  constexpr int NQ = 2 + D;  // gamma, beta, last bias, hidden biases
  float qacc[NQ][NR];
#pragma unroll
  for (int k = 0; k < NQ; ++k)
#pragma unroll
    for (int t = 0; t < NR; ++t) qacc[k][t] = 0.f;
  const bool fuse_w1 = a.w1_part != nullptr;
  float w1acc[OPL][RW_ENC_FIN];
#pragma unroll
  for (int j = 0; j < OPL; ++j)
#pragma unroll
    for (int i = 0; i < RW_ENC_FIN; ++i) w1acc[j][i] = 0.f;
  auto advance = [&](int p) {
    rw_store<NTH>(stg[(p + 1) & 1], buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg[(p + 1) & 1], p + 3);
  };
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t tile = t0 + t;
    const bool active = tile < t1;  // wave-uniform
    const int64_t row = tile * 16 + e;
    const bool ok = active && row < a.rows;
    const int64_t src_row = ok ? row : (active ? tile * 16 : 0);
    uint64_t mask[2] = {0ull, 0ull};  // ReLU derivative of the hidden layers, bit 4 cb + r
    floatx4 acc[1][NB];
    uint4 xf[1][NKH];
    const uint4 x0 = rw_enc_input(a.in0, a.fin, src_row, q, active);
    // the tile's bf16 features (columns >= fin are zero; rows past the end
    // get dz_0 = 0 below) for the fused weight gradient
    if (fuse_w1 && q == 0) *reinterpret_cast<uint2*>(xs + e * RW_ENC_FIN) = make_uint2(x0.x, x0.y);
    rw_enc_first(W0, vb1, x0, ln, acc, &mask[0]);
    {
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[0]) + row * L, q, xf[0], ok);
    }
    int p = 0;
    if constexpr (D == 3) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const int cb = c * RW_CB + cbl;
          const float4 bv = rt_ld4(vbh, cb, q);
          const float b4[4] = {bv.x, bv.y, bv.z, bv.w};
          floatx4& z = acc[0][cb];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = z[r] + b4[r];
            const bool on = v > 0.f;
            mask[1] |= (uint64_t)on << (cb * 4 + r);
            z[r] = on ? v : 0.f;
          }
        }
        __syncthreads();
      }
      p += RW_NC;
      float h[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) h[cb][r] = acc[0][cb][r];
      rt_frags<NB>(h, xf[0]);
      if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[1]) + row * L, q, xf[0], ok);
    }
    // dm: bf16 rows (dL/de^0 of the bf16 edge stream) or fp32 rows
    float dm[NB][4];
    if (a.dm16) {
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {
        float lo[4] = {0.f, 0.f, 0.f, 0.f}, hi[4] = {0.f, 0.f, 0.f, 0.f};
        if (active) rw_unpack(*reinterpret_cast<const uint4*>(a.dm16 + src_row * L + kg * 32 + q * 8), lo, hi);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          dm[2 * kg][r] = ok ? lo[r] : 0.f;
          dm[2 * kg + 1][r] = ok ? hi[r] : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        float4 d4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (active) d4 = rt_ld4(a.dm + src_row * L, cb, q);
        dm[cb][0] = ok ? d4.x : 0.f;
        dm[cb][1] = ok ? d4.y : 0.f;
        dm[cb][2] = ok ? d4.z : 0.f;
        dm[cb][3] = ok ? d4.w : 0.f;
      }
    }
    // last layer + bias: y
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      advance(p + c);
      if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
#pragma unroll
      for (int cbl = 0; cbl < RW_CB; ++cbl) {
        const float4 bv = rt_ld4(vbl, c * RW_CB + cbl, q);
        floatx4& z = acc[0][c * RW_CB + cbl];
        z[0] += bv.x;
        z[1] += bv.y;
        z[2] += bv.z;
        z[3] += bv.w;
      }
      __syncthreads();
    }
    p += RW_NC;
    // LayerNorm recomputed (y becomes xhat), then its backward
    float gv[NB][4];
    if (active) {
      float y[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) y[cb][r] = acc[0][cb][r];
      const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
      float s2 = 0.f;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = y[cb][r] - mu;
          s2 += d * d;
        }
      const float rs = 1.0f / sqrtf(rt_sum4(s2) / L + a.eps);
      float t1s = 0.f, t2s = 0.f;
      {
        float tg[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 g4 = rt_ld4(vg, cb, q);
          const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            y[cb][r] = (y[cb][r] - mu) * rs;
            const float d = dm[cb][r] * g[r];
            t1s += d;
            t2s += d * y[cb][r];
            tg[cb * 4 + r] = dm[cb][r] * y[cb][r];
          }
        }
        t1s = rt_sum4(t1s);
        t2s = rt_sum4(t2s);
        rt_col_totals<NV>(tg, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[0][tt] += tg[tt];
      }
      {
        float tb[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) tb[cb * 4 + r] = dm[cb][r];
        rt_col_totals<NV>(tb, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[1][tt] += tb[tt];
      }
      {
        float tl[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          const float4 g4 = rt_ld4(vg, cb, q);
          const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[cb][r] = rs * (dm[cb][r] * g[r] - t1s / L - y[cb][r] * (t2s / L));
            tl[cb * 4 + r] = gv[cb][r];
          }
        }
        rt_col_totals<NV>(tl, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[2][tt] += tl[tt];
      }
    } else {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) gv[cb][r] = 0.f;
    }
    rt_frags<NB>(gv, xf[0]);
    if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[D - 1]) + row * L, q, xf[0], ok);
    // hidden layers: dz_{j-1} = (dz_j W_j) * [z_{j-1} > 0]
#pragma unroll
    for (int j = D - 1; j >= 1; --j) {
#pragma unroll
      for (int c = 0; c < RW_NC; ++c) {
        advance(p + c);
        if (active) rw_gemm<1>(c, buf + ((p + c) & 1) * RW_CHUNK, xf, acc, ln);
        __syncthreads();
      }
      p += RW_NC;
      if (active) {
        float th[NV];
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            gv[cb][r] = ((mask[j - 1] >> (cb * 4 + r)) & 1ull) ? acc[0][cb][r] : 0.f;
            th[cb * 4 + r] = gv[cb][r];
          }
        rt_col_totals<NV>(th, e);
#pragma unroll
        for (int tt = 0; tt < NR; ++tt) qacc[3 + (j - 1)][tt] += th[tt];
      }
      rt_frags<NB>(gv, xf[0]);
      if (j > 1 || !fuse_w1) {
        if (active) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[j - 1]) + row * L, q, xf[0], ok);
      }
    }
    if (fuse_w1 && active) {
      // dW_1 += dz_0^T x over the tile's 16 rows: dz_0 (bf16, as a stored
      // delta would hold it) through the wave's scratch; lane l forms output
      // rows OPL l .. OPL l + OPL - 1, ascending row order
      {
        uint16_t* dr = dzs + e * Lay::DZS + q * 8;
#pragma unroll
        for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(dr + kg * 32) = rt_to_plain(xf[0][kg]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint2 xv = *reinterpret_cast<const uint2*>(xs + r * RW_ENC_FIN);
        const float x4[4] = {__uint_as_float(xv.x << 16), __uint_as_float(xv.x & 0xffff0000u),
                             __uint_as_float(xv.y << 16), __uint_as_float(xv.y & 0xffff0000u)};
        const uint2 w = *reinterpret_cast<const uint2*>(dzs + r * Lay::DZS + OPL * lane);
        const float d[OPL] = {__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                              __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u)};
#pragma unroll
        for (int j = 0; j < OPL; ++j)
#pragma unroll
          for (int i = 0; i < RW_ENC_FIN; ++i) w1acc[j][i] = fmaf(d[j], x4[i], w1acc[j][i]);
      }
    }
  }
  // column partials: lane (e, q)'s totals are columns 16 cb + 4 q + r for
  // index e * NR + t = 4 cb + r; then the waves in order through LDS (the
  // chunk buffers are free now)
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  {
    float* rw = red + wave * Lay::NVEC;
#pragma unroll
    for (int tt = 0; tt < NR; ++tt) {
      const int i = (lane & 15) * NR + tt;
      const int col = (i >> 2) * 16 + (lane >> 4) * 4 + (i & 3);
#pragma unroll
      for (int h = 0; h < D - 1; ++h) rw[h * L + col] = qacc[3 + h][tt];
      rw[(D - 1) * L + col] = qacc[2][tt];
      rw[D * L + col] = qacc[0][tt];
      rw[(D + 1) * L + col] = qacc[1][tt];
    }
  }
  __syncthreads();
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  for (int i = threadIdx.x; i < Lay::NVEC; i += NTH) {
    float tsum = 0.f;
    for (int w = 0; w < Lay::NWV; ++w) tsum += red[w * Lay::NVEC + i];
    vp[i] = tsum;
  }
  if (fuse_w1) {
    float* wp = a.w1_part + ((int64_t)blockIdx.x * Lay::NWV + wave) * L * a.fin;
#pragma unroll
    for (int j = 0; j < OPL; ++j)
#pragma unroll
      for (int i = 0; i < RW_ENC_FIN; ++i)
        if (i < a.fin) wp[(OPL * lane + j) * a.fin + i] = w1acc[j][i];
  }
}

// Node projections at l = 256 in the streamed-weight form: P[n] = [W_s v_n |
// W_r v_n + b_1] (fp32), v_n the bf16 copy; per 16-row tile of a wave the
// sender then the receiver k-range of the packed W_1 stream through LDS in
// column chunks, and each chunk's accumulators go out as 16-byte row pieces.
struct RwProjLay {
  static constexpr int NWV = 8, NTH = 64 * NWV;
  static constexpr int OFF_BUF = 0;                        // two chunk buffers
  static constexpr int OFF_VEC = 2 * RW_CHUNK * 16;        // b_1
  static constexpr int END = OFF_VEC + RW_L * 4;
  static constexpr int NCH = 2 * RW_NC;
  static_assert(END <= 160 * 1024 && NCH % 2 == 0, "");
};

__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void node_proj_rw_kernel(const uint16_t* __restrict__ V16, int64_t n_local, Lin w1, float* __restrict__ proj) {
  using Lay = RwProjLay;
  constexpr int NTH = Lay::NTH, NKH = RW_NKH, L = RW_L;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* buf = reinterpret_cast<uint4*>(lds + Lay::OFF_BUF);
  float* vb1 = reinterpret_cast<float*>(lds + Lay::OFF_VEC);
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const uint32_t vo_plain = rw_thread_off<false>();
  auto load = [&](RwStage<NTH>& st, int p) {
    // the sender k-range of the packed W_1, then the receiver one
    const int pp = p % Lay::NCH;
    rw_load<NTH, false>(st, RwSrc{w1.wf, 3 * NKH, (1 + pp / RW_NC) * NKH}, pp % RW_NC, vo_plain);
  };
  RwStage<NTH> stg;
  load(stg, 0);
  rw_store<NTH>(stg, buf);
  load(stg, 1);
  rt_copy_vec(vb1, w1.b, L);
  int64_t t0, t1;
  rw_row_tiles(n_local, (int64_t)blockIdx.x * Lay::NWV + wave, (int64_t)gridDim.x * Lay::NWV, t0, t1);
  const int64_t T = (n_local + 15) / 16, Wt = (int64_t)gridDim.x * Lay::NWV;
  const int ntile = (int)((T + Wt - 1) / Wt);
  __syncthreads();
  auto advance = [&](int p) {
    rw_store<NTH>(stg, buf + ((p + 1) & 1) * RW_CHUNK);
    load(stg, p + 2);
  };
  for (int t = 0; t < ntile; ++t) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t tile = t0 + t;
    const bool active = tile < t1;  // wave-uniform
    const int64_t row = tile * 16 + e;
    const bool ok = active && row < n_local;
    const int64_t src_row = ok ? row : (active ? tile * 16 : 0);
    uint4 xv[1][NKH];
#pragma unroll
    for (int kg = 0; kg < NKH; ++kg)
      xv[0][kg] = active ? *reinterpret_cast<const uint4*>(V16 + src_row * L + kg * 32 + q * 8) : make_uint4(0, 0, 0, 0);
    floatx4 acc[1][RW_NB];
#pragma unroll
    for (int side = 0; side < 2; ++side)
#pragma unroll
    for (int c = 0; c < RW_NC; ++c) {
      const int p = side * RW_NC + c;
      advance(p);
      if (active) rw_gemm<1>(c, buf + (p & 1) * RW_CHUNK, xv, acc, ln);
      if (ok) {
        float* op = proj + row * (2 * L) + side * L;
#pragma unroll
        for (int cbl = 0; cbl < RW_CB; ++cbl) {
          const int cb = c * RW_CB + cbl;
          floatx4 z = acc[0][cb];
          if (side) {  // the first Linear's bias rides with the receiver half
            const float4 bv = rt_ld4(vb1, cb, q);
            z[0] += bv.x;
            z[1] += bv.y;
            z[2] += bv.z;
            z[3] += bv.w;
          }
          *reinterpret_cast<float4*>(op + cb * 16 + q * 4) = make_float4(z[0], z[1], z[2], z[3]);
        }
      }
      __syncthreads();
    }
  }
}

template <int L, int KIND>
struct RsRowsLay {
  static constexpr int NKH = L / 32, NB = L / 16;
  static constexpr int W = NB * NKH * 64 * 16;               // one L x L packed layer
  // W_last (fwd), W_last (bwd), then the first Linear: its backward packing
  // for the node half (input 2L), its forward packing for the edge encoder
  static constexpr int W1B = KIND == NODE_BLOCK ? 2 * W : NB * 64 * 16;
  static constexpr int OFF_W1 = 2 * W;
  static constexpr int OFF_SCR = OFF_W1 + W1B;
  static constexpr int SCR = 16 * L * 2;
  static constexpr int END = OFF_SCR + RS_NWV * SCR;
  static constexpr int NVEC = 4 * L;
  static_assert(RS_NWV * NVEC * 4 <= OFF_SCR, "partials reuse the weight area");
};

// Backward of the node half of a block (KIND NODE_BLOCK: input [v | agg],
// residual v + LN(MLP)) or of the edge encoder (ENC_EDGE: input the edge
// features), bf16, depth 2, with the forward recomputed per 16-row tile:
// every wave works alone on its tiles as in the row-split edge kernels.
// Same outputs as rows_bwd_kernel for these kinds.
template <int L, int KIND>
__global__ __launch_bounds__(RS_NTH) void rows_bwd_rs_kernel(RowsBwdArgs a) {
  using Lay = RsRowsLay<L, KIND>;
  constexpr int NKH = Lay::NKH, NB = Lay::NB, W = Lay::W;
  constexpr int NK1 = KIND == NODE_BLOCK ? 2 * NKH : 1;  // k-groups of the first Linear
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* W2f = reinterpret_cast<uint4*>(lds);
  uint4* W2b = reinterpret_cast<uint4*>(lds + W);
  uint4* W1 = reinterpret_cast<uint4*>(lds + Lay::OFF_W1);
  const int wave = wave_id(), lane = threadIdx.x & 63;
  uint16_t* scr = reinterpret_cast<uint16_t*>(lds + Lay::OFF_SCR + wave * Lay::SCR);
  rs_copy_frags(W2f, a.mlp.lin[1].wf, NB, NKH, NKH, 0);
  rs_copy_frags(W2b, a.mlp.lin[1].wb, NB, NKH, NKH, 0);
  if constexpr (KIND == NODE_BLOCK) rs_copy_frags(W1, a.mlp.lin[0].wb, 2 * NB, NKH, NKH, 0);
  else rs_copy_frags(W1, a.mlp.lin[0].wf, NB, 1, 1, 0);
  __syncthreads();
  // column sums of the bias / LayerNorm gradients, folded per tile as in
  // edge_bwd_rs_kernel: hidden bias, last bias, gamma, beta
  constexpr int NG = NB / 4;
  float qacc[4][NG];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int j = 0; j < NG; ++j) qacc[q][j] = 0.f;
  auto fold = [&](int q, float (&t)[NB], int grp) {
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      float x = t[cb];
      x += __shfl_xor(x, 16, 64);
      x += __shfl_xor(x, 32, 64);
#pragma unroll
      for (int j = 0; j < NG; ++j)
        if (cb == grp * NG + j) qacc[q][j] += x;
    }
  };
  const int64_t ntiles = (a.rows + 15) / 16;
  const int64_t nw = (int64_t)gridDim.x * RS_NWV;
  for (int64_t t = (int64_t)blockIdx.x * RS_NWV + wave; t < ntiles; t += nw) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int arow = ln & 15, ach = ln >> 4;
    const int64_t row0 = t * 16;
    const int n = (int)(a.rows - row0 < 16 ? a.rows - row0 : 16);
    // first-layer operands in fragment order (bf16 of the fp32 inputs)
    uint4 xf[NK1];
    if constexpr (KIND == NODE_BLOCK) {
#pragma unroll
      for (int kg = 0; kg < NK1; ++kg) {
        if (kg < NKH && a.in0_16) {  // bf16 copy of v
          xf[kg] = arow < n ? *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a.in0_16) +
                                                              (row0 + arow) * L + kg * 32 + ach * 8)
                            : make_uint4(0, 0, 0, 0);
          continue;
        }
        const float* src = (kg < NKH ? a.in0 : a.in1) + (row0 + arow) * L + (kg % NKH) * 32 + ach * 8;
        float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
        if (arow < n) {
          x0 = reinterpret_cast<const float4*>(src)[0];
          x1 = reinterpret_cast<const float4*>(src)[1];
        }
        uint16_t h[8] = {f2bf(x0.x), f2bf(x0.y), f2bf(x0.z), f2bf(x0.w), f2bf(x1.x), f2bf(x1.y), f2bf(x1.z), f2bf(x1.w)};
        xf[kg] = *reinterpret_cast<const uint4*>(h);
      }
    } else {
      uint16_t h[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = ach * 8 + j;
        h[j] = f2bf((arow < n && k < a.fin) ? a.in0[(row0 + arow) * a.fin + k] : 0.f);
      }
      xf[0] = *reinterpret_cast<const uint4*>(h);
    }
    floatx4 z[NB];
    if constexpr (KIND == NODE_BLOCK) rs_gemm_g<NB, NK1>(xf, a.mlp.lin[0].wf, z, ln);
    else rs_gemm<NB, 1>(xf, W1, z, ln);
    uint32_t mask = 0u;
    float h[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float bv = a.mlp.lin[0].b[cb * 16 + (ln & 15)];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float v = z[cb][r] + bv;
        const bool on = v > 0.f;
        mask |= (on ? 1u : 0u) << (cb * 4 + r);
        h[cb][r] = on ? v : 0.f;
      }
    }
    uint4 hf[NKH];
    rs_to_frags<L>(h, scr, hf, ln);
    rs_store_rows<L>(reinterpret_cast<uint16_t*>(a.hid[0]) + row0 * L, scr, n, ln);
    float y[NB][4];
    {
      floatx4 acc[NB];
      rs_gemm<NB, NKH>(hf, W2f, acc, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float bv = a.mlp.lin[1].b[cb * 16 + (ln & 15)];
#pragma unroll
        for (int r = 0; r < 4; ++r) y[cb][r] = acc[cb][r] + bv;
      }
    }
    float dm[NB][4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = (ln >> 4) * 4 + r;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const int64_t i = (row0 + row) * L + cb * 16 + (ln & 15);
        dm[cb][r] = row < n ? (a.dm16 ? bf2f(a.dm16[i]) : a.dm[i]) : 0.f;
      }
    }
    float mu[4], rs[4], t1[4], t2[4];
    rs_row_totals<NB>(y, mu);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      mu[r] = mu[r] / L;
      float x = 0.f;
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float d = y[cb][r] - mu[r];
        x += d * d;
      }
      rs[r] = x;
    }
    rs_butterfly(rs);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      rs[r] = 1.0f / sqrtf(rs[r] / L + a.eps);
      t1[r] = t2[r] = 0.f;
    }
    {
      float tg[NB], tb[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float g = a.mlp.gamma[cb * 16 + (ln & 15)];
        tg[cb] = tb[cb] = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          y[cb][r] = (y[cb][r] - mu[r]) * rs[r];
          const float d = dm[cb][r] * g;
          t1[r] += d;
          t2[r] += d * y[cb][r];
          tg[cb] += dm[cb][r] * y[cb][r];
          tb[cb] += dm[cb][r];
        }
      }
      fold(2, tg, ln >> 4);
      fold(3, tb, ln >> 4);
    }
    rs_butterfly(t1);
    rs_butterfly(t2);
    float v[NB][4];
    {
      float tl[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float g = a.mlp.gamma[cb * 16 + (ln & 15)];
        tl[cb] = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[cb][r] = rs[r] * (dm[cb][r] * g - t1[r] / L - y[cb][r] * (t2[r] / L));
          tl[cb] += v[cb][r];
        }
      }
      fold(1, tl, ln >> 4);
    }
    uint4 gf[NKH];
    rs_to_frags<L>(v, scr, gf, ln);
    rs_store_rows<L>(reinterpret_cast<uint16_t*>(a.delta[1]) + row0 * L, scr, n, ln);
    {
      floatx4 acc[NB];
      rs_gemm<NB, NKH>(gf, W2b, acc, ln);
      float th[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        th[cb] = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[cb][r] = ((mask >> (cb * 4 + r)) & 1u) ? acc[cb][r] : 0.f;
          th[cb] += v[cb][r];
        }
      }
      fold(0, th, ln >> 4);
    }
    rs_to_frags<L>(v, scr, gf, ln);
    rs_store_rows<L>(reinterpret_cast<uint16_t*>(a.delta[0]) + row0 * L, scr, n, ln);
    if constexpr (KIND == NODE_BLOCK) {
      // input gradients: dv = dm + dz W_1[:, v-block], dagg = dz W_1[:, agg-block]
#pragma unroll
      for (int pass = 0; pass < 2; ++pass) {
        floatx4 acc[NB];
        rs_gemm<NB, NKH>(gf, W1 + pass * NB * NKH * 64, acc, ln);
        float* dst = pass == 0 ? a.dx0 : a.dx1;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = (ln >> 4) * 4 + r;
          if (row < n) {
#pragma unroll
            for (int cb = 0; cb < NB; ++cb) {
              const int64_t o = (row0 + row) * L + cb * 16 + (ln & 15);
              dst[o] = pass == 0 ? acc[cb][r] + a.dm[o] : acc[cb][r];
            }
          }
        }
      }
    }
  }
  // column partials: lane groups, then the waves in order through LDS
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  {
    float* rw = red + wave * Lay::NVEC;
#pragma unroll
    for (int j = 0; j < NG; ++j) {
      const int col = ((lane >> 4) * NG + j) * 16 + (lane & 15);
#pragma unroll
      for (int q = 0; q < 4; ++q) rw[q * L + col] = qacc[q][j];
    }
  }
  __syncthreads();
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  for (int i = threadIdx.x; i < Lay::NVEC; i += RS_NTH) {
    float s = 0.f;
    for (int w = 0; w < RS_NWV; ++w) s += red[w * Lay::NVEC + i];
    vp[i] = s;
  }
}

// ------------------------------------------------ row MLPs in T form ---
// Encoders and the node half of a block (bf16, depth 2, l in {64, 128}) with
// the T-form products of the edge kernels: one wave per 16-row tile, no LDS
// round trips, weights and vectors in LDS.  The first Linear's B operand is
// the input row tile in plain order: the edge / node features (fin <= 16
// values, lane groups 0 and 1) or [v | agg] (2 l values).
template <int L, int KIND>
struct RtRowsLay {
  static constexpr int NKH = L / 32, NB = L / 16;
  static constexpr int W = NB * NKH * 64 * 16;           // one l x l packed layer
  static constexpr int NK1 = KIND == NODE_BLOCK ? 2 * NKH : 1;
  static constexpr int W1 = NB * NK1 * 64 * 16;          // first Linear (forward packing)
  // forward: W1, W2, then b1, b2, gamma, beta
  static constexpr int F_W2 = W1, F_VEC = W1 + W, F_END = F_VEC + 4 * L * 4;
  // backward: W2 (fwd), W2 (bwd), then W1 (ENC_EDGE: forward packing, for the
  // recompute; NODE_BLOCK: backward packing, both input blocks), then b1, b2, gamma
  static constexpr int B_W2F = 0, B_W2B = W, B_W1 = 2 * W;
  static constexpr int B_W1S = KIND == NODE_BLOCK ? 2 * W : W1;
  static constexpr int B_VEC = B_W1 + B_W1S, B_END = B_VEC + 3 * L * 4;
  // waves per workgroup: forward 16 (at most 128 registers), backward 12 (168)
  static constexpr int FNWV = 16, FNTH = 64 * FNWV, NWV = 12, NTH = 64 * NWV;
  static constexpr int NVEC = 4 * L;                     // bias / LayerNorm partials per wave
  // ENC_EDGE with the fused first-Linear weight gradient: per-wave scratch
  // for a tile's dz_0 (16 rows of L bf16, 8 columns of padding) and features
  // (16 rows of W1_FIN bf16)
  static constexpr int W1_FIN = 4, DZS = L + 8;
  static constexpr int B_SCR = B_END, SCR = 16 * DZS * 2 + 16 * W1_FIN * 2;
  static constexpr int B_END_W1 = KIND == ENC_EDGE ? B_SCR + NWV * SCR : B_END;
  static_assert(F_END <= 160 * 1024 && B_END <= 160 * 1024 && B_END_W1 <= 160 * 1024, "LDS");
  static_assert(NWV * NVEC * 4 <= B_VEC, "partials reuse the weight area");
};

// First-Linear B operand of a row tile (row `row`, lane group q).
template <int L, int KIND>
__device__ __forceinline__ void rt_rows_input(const float* __restrict__ in0, const float* __restrict__ in1,
                                              const uint16_t* __restrict__ in0_16, int fin, int64_t row, int q,
                                              uint4 (&xf)[RtRowsLay<L, KIND>::NK1]) {
  constexpr int NKH = L / 32;
  if constexpr (KIND == NODE_BLOCK) {
#pragma unroll
    for (int kg = 0; kg < 2 * NKH; ++kg) {
      if (kg < NKH && in0_16) {  // bf16 copy of v (the rounded operand)
        xf[kg] = *reinterpret_cast<const uint4*>(in0_16 + row * L + kg * 32 + q * 8);
        continue;
      }
      const float* src = (kg < NKH ? in0 : in1) + row * L + (kg % NKH) * 32 + q * 8;
      const float4 x0 = reinterpret_cast<const float4*>(src)[0], x1 = reinterpret_cast<const float4*>(src)[1];
      xf[kg] = make_uint4(bf_pack(x0.x, x0.y), bf_pack(x0.z, x0.w), bf_pack(x1.x, x1.y), bf_pack(x1.z, x1.w));
    }
  } else {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = q * 8 + j;
      x[j] = k < fin ? in0[row * fin + k] : 0.f;
    }
    xf[0] = make_uint4(bf_pack(x[0], x[1]), bf_pack(x[2], x[3]), bf_pack(x[4], x[5]), bf_pack(x[6], x[7]));
  }
}

// acc += b (a T-order vector in LDS), then ReLU; bits of the mask, T-form frags.
template <int NB>
__device__ __forceinline__ void rt_bias_relu(floatx4 (&z)[NB], const float* bv, int q, float (&h)[NB][4],
                                             uint32_t* mask) {
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) {
    const float4 b = rt_ld4(bv, cb, q);
    const float b4[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v = z[cb][r] + b4[r];
      const bool on = v > 0.f;
      if (mask) *mask |= (on ? 1u : 0u) << (cb * 4 + r);
      h[cb][r] = on ? v : 0.f;
    }
  }
}

// Forward: ENC_EDGE -> bf16 rows; ENC_NODE -> fp32 rows + bf16 copy;
// NODE_BLOCK -> v + LN(MLP([v | agg])) fp32 + bf16 copy, and the ReLU output
// of the first Linear (bf16, for the backward) when a.hid_out is set (only
// that when a.out is null).
template <int L, int KIND>
__global__ __launch_bounds__((RtRowsLay<L, KIND>::FNTH)) void rows_rt_fwd_kernel(RowsFwdArgs a) {
  using Lay = RtRowsLay<L, KIND>;
  constexpr int NKH = Lay::NKH, NB = Lay::NB, NK1 = Lay::NK1;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* W1 = reinterpret_cast<uint4*>(lds);
  uint4* W2 = reinterpret_cast<uint4*>(lds + Lay::F_W2);
  float* vb1 = reinterpret_cast<float*>(lds + Lay::F_VEC);
  float* vb2 = vb1 + L;
  float* vg = vb1 + 2 * L;
  float* vbt = vb1 + 3 * L;
  rs_copy_frags(W1, a.mlp.lin[0].wf, NB, NK1, NK1, 0);
  rt_copy_frags(W2, a.mlp.lin[1].wf, NB, NKH, NKH, 0);
  rt_copy_vec(vb1, a.mlp.lin[0].b, L);
  rt_copy_vec(vb2, a.mlp.lin[1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  rt_copy_vec(vbt, a.mlp.beta, L);
  __syncthreads();
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int64_t ntiles = (a.rows + 15) / 16;
  for (int64_t t = (int64_t)blockIdx.x * Lay::FNWV + wave; t < ntiles; t += (int64_t)gridDim.x * Lay::FNWV) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t row = t * 16 + e;
    const bool ok = row < a.rows;
    const int64_t src = ok ? row : t * 16;  // rows past the end repeat the tile's first row (not stored)
    uint4 xf[NK1];
    rt_rows_input<L, KIND>(a.in0, a.in1, reinterpret_cast<const uint16_t*>(a.in0_16), a.fin, src, q, xf);
    floatx4 z[NB];
    rt_gemm<NB, NK1>(W1, xf, z, ln);
    float h[NB][4];
    rt_bias_relu<NB>(z, vb1, q, h, nullptr);
    uint4 hf[NKH];
    rt_frags<NB>(h, hf);
    if constexpr (KIND == NODE_BLOCK) {
      if (a.hid_out) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid_out) + row * L, q, hf, ok);
      if (!a.out) continue;  // only the ReLU output wanted (the backward's recompute)
    }
    floatx4 acc[NB];
    rt_gemm<NB, NKH>(W2, hf, acc, ln);
    float y[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 bv = rt_ld4(vb2, cb, q);
      y[cb][0] = acc[cb][0] + bv.x;
      y[cb][1] = acc[cb][1] + bv.y;
      y[cb][2] = acc[cb][2] + bv.z;
      y[cb][3] = acc[cb][3] + bv.w;
    }
    const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
    float dv[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float d = y[cb][r] - mu;
        dv[cb][r] = d * d;
      }
    const float rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 g = rt_ld4(vg, cb, q), bt = rt_ld4(vbt, cb, q);
      y[cb][0] = g.x * ((y[cb][0] - mu) * rs) + bt.x;
      y[cb][1] = g.y * ((y[cb][1] - mu) * rs) + bt.y;
      y[cb][2] = g.z * ((y[cb][2] - mu) * rs) + bt.z;
      y[cb][3] = g.w * ((y[cb][3] - mu) * rs) + bt.w;
    }
    if constexpr (KIND == NODE_BLOCK) {  // residual: v + m
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 v = rt_ld4(a.in0 + src * L, cb, q);
        y[cb][0] = y[cb][0] + v.x;
        y[cb][1] = y[cb][1] + v.y;
        y[cb][2] = y[cb][2] + v.z;
        y[cb][3] = y[cb][3] + v.w;
      }
    }
    uint4 o[NKH];
    rt_frags<NB>(y, o);
    if constexpr (KIND == ENC_EDGE) {
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.out) + row * L, q, o, ok);
    } else {
      if (ok) {
        float* op = reinterpret_cast<float*>(a.out) + row * L;
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
          *reinterpret_cast<float4*>(op + cb * 16 + q * 4) = make_float4(y[cb][0], y[cb][1], y[cb][2], y[cb][3]);
      }
      if (a.out16) rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.out16) + row * L, q, o, ok);
    }
  }
}

// Backward: ENC_NODE / ENC_EDGE recompute their tile's forward from the features;
// NODE_BLOCK takes the first Linear's ReLU output from the forward
// (a.hid_in) and ends in the input gradients dv = dm + dz W_1[:, v-block],
// dagg = dz W_1[:, agg-block].  Outputs as rows_bwd_kernel for these kinds.
template <int L, int KIND>
__global__ __launch_bounds__((RtRowsLay<L, KIND>::NTH)) void rows_rt_bwd_kernel(RowsBwdArgs a) {
  using Lay = RtRowsLay<L, KIND>;
  constexpr int NKH = Lay::NKH, NB = Lay::NB, NK1 = Lay::NK1, W = Lay::W;
  constexpr int NV = 4 * NB, NR = NV / 16;
  extern __shared__ __align__(16) unsigned char lds[];
  uint4* W2f = reinterpret_cast<uint4*>(lds + Lay::B_W2F);
  uint4* W2b = reinterpret_cast<uint4*>(lds + Lay::B_W2B);
  uint4* W1 = reinterpret_cast<uint4*>(lds + Lay::B_W1);
  float* vb1 = reinterpret_cast<float*>(lds + Lay::B_VEC);
  float* vb2 = vb1 + L;
  float* vg = vb1 + 2 * L;
  rt_copy_frags(W2f, a.mlp.lin[1].wf, NB, NKH, NKH, 0);
  rt_copy_frags(W2b, a.mlp.lin[1].wb, NB, NKH, NKH, 0);
  if constexpr (KIND == NODE_BLOCK) rt_copy_frags(W1, a.mlp.lin[0].wb, 2 * NB, NKH, NKH, 0);
  else rs_copy_frags(W1, a.mlp.lin[0].wf, NB, NK1, NK1, 0);
  rt_copy_vec(vb1, a.mlp.lin[0].b, L);
  rt_copy_vec(vb2, a.mlp.lin[1].b, L);
  rt_copy_vec(vg, a.mlp.gamma, L);
  __syncthreads();
  const int wave = wave_id(), lane = threadIdx.x & 63;
  // column totals (rt_col_totals' share of each lane): hidden bias, last bias, gamma, beta
  float qacc[4][NR];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int t = 0; t < NR; ++t) qacc[k][t] = 0.f;
  auto coltot = [&](float (&x)[NB][4], int k, int e) {
    float* f = &x[0][0];
    rt_col_totals<NV>(*reinterpret_cast<float(*)[NV]>(f), e);
#pragma unroll
    for (int t = 0; t < NR; ++t) qacc[k][t] += f[t];
  };
  // fused first-Linear weight gradient (ENC_EDGE, fin <= W1_FIN): lane l
  // accumulates dW_1 rows OPL l .. OPL l + OPL - 1, columns 0 .. W1_FIN - 1
  constexpr int OPL = L / 64;
  const bool fuse_w1 = KIND == ENC_EDGE && a.w1_part != nullptr;
  uint16_t* dz = reinterpret_cast<uint16_t*>(lds + Lay::B_SCR + wave * Lay::SCR);
  uint16_t* xs = dz + 16 * Lay::DZS;
  float w1acc[OPL][4];
#pragma unroll
  for (int j = 0; j < OPL; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) w1acc[j][i] = 0.f;
  const int64_t ntiles = (a.rows + 15) / 16;
  for (int64_t t = (int64_t)blockIdx.x * Lay::NWV + wave; t < ntiles; t += (int64_t)gridDim.x * Lay::NWV) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int e = ln & 15, q = ln >> 4;
    const int64_t row = t * 16 + e;
    const bool ok = row < a.rows;
    const int64_t src = ok ? row : t * 16;
    uint32_t mask = 0u;
    uint4 hf[NKH];
    if constexpr (KIND == NODE_BLOCK) {
      // h_1 of the forward (plain order) -> T order; its sign is the ReLU mask
      rt_load_relu<NKH>(reinterpret_cast<const uint16_t*>(a.hid_in) + src * L, q, hf, mask);
    } else {
      uint4 xf[NK1];
      rt_rows_input<L, KIND>(a.in0, a.in1, nullptr, a.fin, src, q, xf);
      // the tile's bf16 features (columns >= fin are zero) for the fused
      // weight gradient; rows past the end get dz_0 = 0 below
      if (fuse_w1 && q == 0) *reinterpret_cast<uint2*>(xs + e * Lay::W1_FIN) = make_uint2(xf[0].x, xf[0].y);
      floatx4 z[NB];
      rt_gemm<NB, NK1>(W1, xf, z, ln);
      float h[NB][4];
      rt_bias_relu<NB>(z, vb1, q, h, &mask);
      rt_frags<NB>(h, hf);
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.hid[0]) + row * L, q, hf, ok);
    }
    float y[NB][4];
    {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(W2f, hf, acc, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 bv = rt_ld4(vb2, cb, q);
        y[cb][0] = acc[cb][0] + bv.x;
        y[cb][1] = acc[cb][1] + bv.y;
        y[cb][2] = acc[cb][2] + bv.z;
        y[cb][3] = acc[cb][3] + bv.w;
      }
    }
    float dm[NB][4];
    if (a.dm16) {
      // bf16 rows (dL/de^0 of the bf16 edge stream), plain order -> T order
#pragma unroll
      for (int kg = 0; kg < NKH; ++kg) {
        const uint4 t = rt_from_plain(*reinterpret_cast<const uint4*>(a.dm16 + src * L + kg * 32 + q * 8));
        const uint32_t w[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {  // dword i: block 2 kg + i / 2, columns 2 (i % 2) .. + 1
          dm[2 * kg + i / 2][2 * (i % 2)] = ok ? __uint_as_float(w[i] << 16) : 0.f;
          dm[2 * kg + i / 2][2 * (i % 2) + 1] = ok ? __uint_as_float(w[i] & 0xffff0000u) : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 d4 = rt_ld4(a.dm + src * L, cb, q);
        dm[cb][0] = ok ? d4.x : 0.f;
        dm[cb][1] = ok ? d4.y : 0.f;
        dm[cb][2] = ok ? d4.z : 0.f;
        dm[cb][3] = ok ? d4.w : 0.f;
      }
    }
    // LayerNorm (recomputed): y becomes xhat
    const float mu = rt_sum4(rt_lane_sum<NB>(y)) / L;
    float rs;
    {
      float dv[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = y[cb][r] - mu;
          dv[cb][r] = d * d;
        }
      rs = 1.0f / sqrtf(rt_sum4(rt_lane_sum<NB>(dv)) / L + a.eps);
    }
    // LayerNorm backward: dy = rstd (dm g - mean(dm g) - xhat mean(dm g xhat))
    float t1, t2;
    {
      float p1[4], p2[4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const float4 g4 = rt_ld4(vg, cb, q);
        const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          y[cb][r] = (y[cb][r] - mu) * rs;
          const float d = dm[cb][r] * g[r];
          p1[r] = cb == 0 ? d : p1[r] + d;
          p2[r] = cb == 0 ? d * y[cb][r] : p2[r] + d * y[cb][r];
        }
      }
      t1 = rt_sum4((p1[0] + p1[1]) + (p1[2] + p1[3]));
      t2 = rt_sum4((p2[0] + p2[1]) + (p2[2] + p2[3]));
    }
    float v[NB][4];
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) {
      const float4 g4 = rt_ld4(vg, cb, q);
      const float g[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        v[cb][r] = rs * (dm[cb][r] * g[r] - t1 / L - y[cb][r] * (t2 / L));
        y[cb][r] = dm[cb][r] * y[cb][r];  // gamma's column terms
      }
    }
    coltot(y, 2, e);   // gamma
    coltot(dm, 3, e);  // beta
    uint4 gf[NKH];
    rt_frags<NB>(v, gf);
    rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[1]) + row * L, q, gf, ok);
    coltot(v, 1, e);  // last bias
    {
      floatx4 acc[NB];
      rt_gemm<NB, NKH>(W2b, gf, acc, ln);
#pragma unroll
      for (int cb = 0; cb < NB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) v[cb][r] = ((mask >> (cb * 4 + r)) & 1u) ? acc[cb][r] : 0.f;
    }
    rt_frags<NB>(v, gf);
    if (fuse_w1) {
      // dW_1 += dz_0^T x over the tile's 16 rows: dz_0 (bf16, as a stored
      // delta would hold it) through the wave's scratch, then lane l forms
      // output rows OPL l .. OPL l + OPL - 1, ascending row order
      {
        uint16_t* dr = dz + e * Lay::DZS + q * 8;
#pragma unroll
        for (int kg = 0; kg < NKH; ++kg) *reinterpret_cast<uint4*>(dr + kg * 32) = rt_to_plain(gf[kg]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint2 xv = *reinterpret_cast<const uint2*>(xs + r * Lay::W1_FIN);
        const float x4[4] = {__uint_as_float(xv.x << 16), __uint_as_float(xv.x & 0xffff0000u),
                             __uint_as_float(xv.y << 16), __uint_as_float(xv.y & 0xffff0000u)};
        float d[OPL];
        if constexpr (OPL == 2) {
          const uint32_t w = *reinterpret_cast<const uint32_t*>(dz + r * Lay::DZS + 2 * lane);
          d[0] = __uint_as_float(w << 16);
          d[1] = __uint_as_float(w & 0xffff0000u);
        } else {
          d[0] = __uint_as_float((uint32_t)dz[r * Lay::DZS + lane] << 16);
        }
#pragma unroll
        for (int j = 0; j < OPL; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) w1acc[j][i] = fmaf(d[j], x4[i], w1acc[j][i]);
      }
    } else {
      rt_store_frags<NKH>(reinterpret_cast<uint16_t*>(a.delta[0]) + row * L, q, gf, ok);
    }
    coltot(v, 0, e);  // hidden bias
    if constexpr (KIND == NODE_BLOCK) {
#pragma unroll
      for (int pass = 0; pass < 2; ++pass) {
        floatx4 acc[NB];
        rt_gemm<NB, NKH>(W1 + pass * NB * NKH * 64, gf, acc, ln);
        if (pass == 0) {  // dv = dz W_1[:, v-block] + dm
#pragma unroll
          for (int cb = 0; cb < NB; ++cb) {
            const float4 d4 = rt_ld4(a.dm + src * L, cb, q);
            acc[cb][0] += d4.x;
            acc[cb][1] += d4.y;
            acc[cb][2] += d4.z;
            acc[cb][3] += d4.w;
          }
        }
        if (ok) {
          float* op = (pass == 0 ? a.dx0 : a.dx1) + row * L;
#pragma unroll
          for (int cb = 0; cb < NB; ++cb)
            *reinterpret_cast<float4*>(op + cb * 16 + q * 4) = make_float4(acc[cb][0], acc[cb][1], acc[cb][2], acc[cb][3]);
        }
      }
    }
  }
  // column partials: lane (e, q)'s totals are columns 16 cb + 4 q + r for
  // index e * NR + t = 4 cb + r; then the waves in order through LDS
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  {
    float* rw = red + wave * Lay::NVEC;
#pragma unroll
    for (int t = 0; t < NR; ++t) {
      const int i = (lane & 15) * NR + t;
      const int col = (i >> 2) * 16 + (lane >> 4) * 4 + (i & 3);
#pragma unroll
      for (int k = 0; k < 4; ++k) rw[k * L + col] = qacc[k][t];
    }
  }
  __syncthreads();
  float* vp = a.vpart + (int64_t)blockIdx.x * a.nvec;
  for (int i = threadIdx.x; i < Lay::NVEC; i += Lay::NTH) {
    float s = 0.f;
    for (int w = 0; w < Lay::NWV; ++w) s += red[w * Lay::NVEC + i];
    vp[i] = s;
  }
  if (fuse_w1) {
    float* wp = a.w1_part + ((int64_t)blockIdx.x * Lay::NWV + wave) * L * a.fin;
#pragma unroll
    for (int j = 0; j < OPL; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (i < a.fin) wp[(OPL * lane + j) * a.fin + i] = w1acc[j][i];
  }
}

// --------------------------------------------------- node input gradient ---
// Gradient reaching the nodes through the first Linear of a block's edge MLP.
// Its sender and receiver column blocks W_s, W_r are shared by all edges, so
//   dv[n] += dzr[n] W_r + dzs[n] W_s   (owned n)
//   dh[n - n_owned] = dzs[n] W_s       (halo n)
// with dzr[n] the sum of dz_0 over the edges n receives (from the edge
// backward kernel) and dzs[n] the sum over the edges n sends, gathered here in
// ascending local edge id through the transposed CSR.  Sums are fp32; in
// bf16 mode each fp32 operand enters the bf16 products as hi + lo, two bf16
// values whose sum is within 2^-17 of it (relative).
template <class P, int L>
struct InGradTile {
  static constexpr int TM = 32;                                      // nodes per workgroup
  static constexpr int LDT = L + P::PAD;
  static constexpr int NOP = sizeof(typename P::T) == 2 ? 4 : 2;     // operand tiles: (hi, lo) x (r, s)
  static constexpr int END = NOP * TM * LDT * (int)sizeof(typename P::T);
};

template <class P>
__device__ __forceinline__ void put_operand(typename P::T* hi, typename P::T* lo, float x) {
  if constexpr (sizeof(typename P::T) == 2) {
    const uint16_t h = f2bf(x);
    *hi = h;
    *lo = f2bf(x - bf2f(h));
  } else {
    *hi = x;
  }
}

template <int P_, int L>
__global__ __launch_bounds__(NT) void input_grad_kernel(InGradArgs a) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  using G = InGradTile<P, L>;
  constexpr int TM = G::TM, LDT = G::LDT, MB = TM / 16;
  constexpr int NBW = L / 16 / NW;
  constexpr int NKH = L / P::KG;
  constexpr bool SPLIT = sizeof(T) == 2;
  extern __shared__ __align__(16) unsigned char lds[];
  T* Rh = reinterpret_cast<T*>(lds);
  T* Sh = Rh + TM * LDT;
  T* Rl = SPLIT ? Sh + TM * LDT : Rh;
  T* Sl = SPLIT ? Rl + TM * LDT : Sh;
  const int64_t n0 = (int64_t)blockIdx.x * TM;
  const int tid = threadIdx.x, wave = tid >> 6;
  const T* dz = reinterpret_cast<const T*>(a.dz);
  // sender sums: (node, 16-byte chunk) items, ascending edges, 4 loads in
  // flight; or, when they were formed chunk by chunk (sender_sums_kernel),
  // read back from dzs
  constexpr int E16 = 16 / sizeof(T);
  constexpr int CPR = L / E16;
  if (a.dzs_ready) {
    for (int it = tid; it < TM * (L / 4); it += NT) {
      const int row = it / (L / 4), c = (it % (L / 4)) * 4;
      const int64_t node = n0 + row;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (node < a.n_local) v = *reinterpret_cast<const float4*>(a.dzs + node * L + c);
      put_operand<P>(Sh + row * LDT + c, Sl + row * LDT + c, v.x);
      put_operand<P>(Sh + row * LDT + c + 1, Sl + row * LDT + c + 1, v.y);
      put_operand<P>(Sh + row * LDT + c + 2, Sl + row * LDT + c + 2, v.z);
      put_operand<P>(Sh + row * LDT + c + 3, Sl + row * LDT + c + 3, v.w);
    }
  }
  // receiver sums (owned rows; zero for halo rows and past the end): this
  // thread's rows are loaded before the sender gather, so that their latency
  // overlaps it, and go to LDS after it
  constexpr int RPT = TM * (L / 4) / NT;  // 16-byte receiver chunks per thread
  static_assert(TM * (L / 4) % NT == 0, "receiver chunks");
  float4 rv[RPT];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int it = tid + k * NT, row = it / (L / 4), c = (it % (L / 4)) * 4;
    const int64_t node = n0 + row;
    // rows past the owned ones read row 0 (then replaced by zeros)
    rv[k] = a.n_owned > 0 ? *reinterpret_cast<const float4*>(a.dzr + (node < a.n_owned ? node : 0) * L + c)
                          : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  for (int it = tid; !a.dzs_ready && it < TM * CPR; it += NT) {
    const int row = it / CPR, c = (it % CPR) * E16;
    const int64_t node = n0 + row;
    float s[E16];
#pragma unroll
    for (int j = 0; j < E16; ++j) s[j] = 0.f;
    if (node < a.n_local) {
      // up to IG_FLIGHT rows in flight per thread, summed in ascending edge
      // order: the group's edge ids are loaded first, then its rows, each
      // all at once (positions past the end repeat the last edge, a cache
      // hit, and are not summed)
      constexpr int IG_FLIGHT = 16;
      const int32_t end = a.trow[node + 1];
      for (int32_t i = a.trow[node]; i < end; i += IG_FLIGHT) {
        int32_t id[IG_FLIGHT];
#pragma unroll
        for (int u = 0; u < IG_FLIGHT; ++u) id[u] = a.tedge[i + u < end ? i + u : end - 1];
        uint4 v[IG_FLIGHT];
#pragma unroll
        for (int u = 0; u < IG_FLIGHT; ++u) v[u] = *reinterpret_cast<const uint4*>(dz + (int64_t)id[u] * L + c);
#pragma unroll
        for (int u = 0; u < IG_FLIGHT; ++u) {
          if (i + u < end) {
            const T* t = reinterpret_cast<const T*>(&v[u]);
#pragma unroll
            for (int j = 0; j < E16; ++j) s[j] += to_f(t[j]);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < E16; ++j) put_operand<P>(Sh + row * LDT + c + j, Sl + row * LDT + c + j, s[j]);
    if (node < a.n_local) {
#pragma unroll
      for (int j = 0; j < E16; j += 4)
        *reinterpret_cast<float4*>(a.dzs + node * L + c + j) = make_float4(s[j], s[j + 1], s[j + 2], s[j + 3]);
    }
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int it = tid + k * NT, row = it / (L / 4), c = (it % (L / 4)) * 4;
    const float4 v = n0 + row < a.n_owned ? rv[k] : make_float4(0.f, 0.f, 0.f, 0.f);
    put_operand<P>(Rh + row * LDT + c, Rl + row * LDT + c, v.x);
    put_operand<P>(Rh + row * LDT + c + 1, Rl + row * LDT + c + 1, v.y);
    put_operand<P>(Rh + row * LDT + c + 2, Rl + row * LDT + c + 2, v.z);
    put_operand<P>(Rh + row * LDT + c + 3, Rl + row * LDT + c + 3, v.w);
  }
  __syncthreads();
  const int nb = wave * NBW;
  floatx4 acc[MB][NBW];
  wave_gemm_k<P, MB, NBW, NKH, true>(Rh, LDT, a.w1.wb, 2 * (L / 16) + nb, acc);
  if constexpr (SPLIT) wave_gemm_k<P, MB, NBW, NKH, false>(Rl, LDT, a.w1.wb, 2 * (L / 16) + nb, acc);
  wave_gemm_k<P, MB, NBW, NKH, false>(Sh, LDT, a.w1.wb, (L / 16) + nb, acc);
  if constexpr (SPLIT) wave_gemm_k<P, MB, NBW, NKH, false>(Sl, LDT, a.w1.wb, (L / 16) + nb, acc);
  // the dv values this lane adds to, all loaded before any is written (rows
  // past the owned ones read row 0 and are not written)
  float old[MB][4][NBW];
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t node = n0 + m * 16 + acc_row(r);
#pragma unroll
      for (int nn = 0; nn < NBW; ++nn)
        old[m][r][nn] = a.n_owned > 0 ? a.dv[(node < a.n_owned ? node : 0) * L + (nb + nn) * 16 + acc_col()] : 0.f;
    }
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t node = n0 + m * 16 + acc_row(r);
#pragma unroll
      for (int nn = 0; nn < NBW; ++nn) {
        const int col = (nb + nn) * 16 + acc_col();
        if (node < a.n_owned) {
          a.dv[node * L + col] = old[m][r][nn] + acc[m][nn][r];
        } else if (node < a.n_local && a.dh) {
          a.dh[(node - a.n_owned) * L + col] = acc[m][nn][r];
        }
      }
    }
}

// Per-sender sums of dz_0 over the edges of one chunk [e_lo, e_hi) (dz rows
// stored from e_lo): dzs[n] = (first chunk ? 0 : dzs[n]) + sum, each node's
// edges of the chunk in ascending id (a contiguous run of its transposed-CSR
// list).  Chunk by chunk this gives the sums input_grad_kernel forms in one
// pass when the whole edge range is one chunk.
template <int P_, int L>
__global__ __launch_bounds__(NT) void sender_sums_kernel(const int32_t* __restrict__ trow,
                                                         const int32_t* __restrict__ tedge, const void* dzv,
                                                         int64_t e_lo, int64_t e_hi, int64_t n_local,
                                                         float* __restrict__ dzs, int first,
                                                         const int32_t* __restrict__ range) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  constexpr int E16 = 16 / sizeof(T);
  constexpr int CPR = L / E16;
  const T* dz = reinterpret_cast<const T*>(dzv);
  // every local node, or (range) only the senders [range[0], range[1]] of
  // the edges in [e_lo, e_hi): the other nodes' sums do not change
  const int64_t n0 = range ? (int64_t)range[0] : 0;
  const int64_t n1 = range ? (int64_t)range[1] + 1 : n_local;
  for (int64_t it = (int64_t)blockIdx.x * NT + threadIdx.x; it < (n1 - n0) * CPR; it += (int64_t)gridDim.x * NT) {
    const int64_t node = n0 + it / CPR;
    const int c = (int)(it % CPR) * E16;
    int32_t lo = trow[node], hi = trow[node + 1];
    while (lo < hi) {  // first of the node's edges at or after e_lo
      const int32_t mid = (lo + hi) >> 1;
      if (tedge[mid] < e_lo) lo = mid + 1;
      else hi = mid;
    }
    float s[E16];
#pragma unroll
    for (int j = 0; j < E16; ++j) s[j] = 0.f;
    // up to 16 rows in flight, summed in ascending edge order; the group's
    // edge ids load at once (positions past the node's end re-read its last
    // id and are then marked past every chunk)
    const int32_t nend = trow[node + 1];
    for (int32_t i = lo; i < nend; i += 16) {
      int32_t ed[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) ed[u] = tedge[i + u < nend ? i + u : nend - 1];
#pragma unroll
      for (int u = 0; u < 16; ++u) ed[u] = i + u < nend ? ed[u] : INT32_MAX;
      uint4 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        v[u] = ed[u] < e_hi ? *reinterpret_cast<const uint4*>(dz + (int64_t)(ed[u] - e_lo) * L + c)
                            : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (ed[u] < e_hi) {
          const T* t = reinterpret_cast<const T*>(&v[u]);
#pragma unroll
          for (int j = 0; j < E16; ++j) s[j] += to_f(t[j]);
        }
      }
      if (ed[15] >= e_hi) break;
    }
    float* d = dzs + node * L + c;
#pragma unroll
    for (int j = 0; j < E16; ++j) d[j] = (first ? 0.f : d[j]) + s[j];
  }
}

// range[0] = min, range[1] = max of send[e_lo .. e_hi) (range pre-filled
// with INT32_MAX, -1); integer minimum and maximum, so the result does not
// depend on the order of the updates.
__global__ __launch_bounds__(NT) void sender_range_kernel(const int32_t* __restrict__ send, int64_t e_lo, int64_t e_hi,
                                                          int32_t* __restrict__ range) {
  int32_t lo = INT32_MAX, hi = -1;
  for (int64_t e = e_lo + (int64_t)blockIdx.x * NT + threadIdx.x; e < e_hi; e += (int64_t)gridDim.x * NT) {
    const int32_t v = send[e];
    lo = v < lo ? v : lo;
    hi = v > hi ? v : hi;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int32_t a = __shfl_xor(lo, off, 64), b = __shfl_xor(hi, off, 64);
    lo = a < lo ? a : lo;
    hi = b > hi ? b : hi;
  }
  if ((threadIdx.x & 63) == 0 && hi >= 0) {
    atomicMin(range, lo);
    atomicMax(range + 1, hi);
  }
}

// -------------------------------------------------- weight gradients ---
// part[s][o][i] = sum over rows of split s of delta[row][o] * A[row][i], as an
// MFMA GEMM with both operands staged transposed in LDS (rows contiguous).
constexpr int DW_TO = 128, DW_TI = 128, DW_RC = 64;

// EL consecutive elements (16 bytes of storage type) of row `row` of the
// weight-gradient input operand, starting at column col, as storage type.
template <class P>
__device__ __forceinline__ uint4 dw_load_a(const DwArgs& a, int64_t row, int col) {
  using T = typename P::T;
  T v[P::EL];
  if (a.a_kind == 0) {
    return *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.a0) + row * a.lda0 + col);
  } else if (a.a_kind == 1) {
    const float* src = reinterpret_cast<const float*>(a.a0) + row * a.lda0 + col;
#pragma unroll
    for (int e = 0; e < P::EL; ++e) v[e] = P::cvt((col + e < a.lda0) ? src[e] : 0.f);
  } else if (a.a_kind == 2) {
    const int L = a.L;
    if (col < L) return *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.a0) + row * L + col);
    const int64_t node = col < 2 * L ? (int64_t)a.send[row] : (int64_t)a.erecv[row];
    const int c = col < 2 * L ? col - L : col - 2 * L;
    if (a.a3) {  // bf16 copy of the node rows, owned then halo
      return *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.a3) + node * L + c);
    }
    const float* src = node < a.n_owned ? a.a1 + node * L + c : a.a2 + (node - a.n_owned) * L + c;
#pragma unroll
    for (int e = 0; e < P::EL; ++e) v[e] = P::cvt(src[e]);
  } else if (a.a_kind == 3) {
    const int L = a.L;
    const float* src = (col < L ? reinterpret_cast<const float*>(a.a0) + row * L + col : a.a1 + row * L + (col - L));
#pragma unroll
    for (int e = 0; e < P::EL; ++e) v[e] = P::cvt(src[e]);
  } else if (a.a_kind == 5) {
    // node concat with v as bf16 rows (bf16 mode; EL = 8 columns never straddle v | agg)
    const int L = a.L;
    if (col < L) return *reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(a.a3) + row * L + col);
    const float* src = a.a1 + row * L + (col - L);
#pragma unroll
    for (int e = 0; e < P::EL; ++e) v[e] = P::cvt(src[e]);
  } else {
    // node rows, fp32: owned rows from a0, halo rows from a2
    const float* src = row < a.n_owned ? reinterpret_cast<const float*>(a.a0) + row * a.lda0 + col
                                       : a.a2 + (row - a.n_owned) * a.lda0 + col;
#pragma unroll
    for (int e = 0; e < P::EL; ++e) v[e] = P::cvt(src[e]);
  }
  return *reinterpret_cast<const uint4*>(v);
}

// Transposed LDS tiles [column][row] of DW_RC rows.  A wave stores 16 rows
// of four column groups (EL columns each) at once.  In fp32 the row padding
// alone spreads them over the banks; in bf16 the four groups' columns are
// 8 apart, which the padding maps onto the same banks, so the row index is
// XORed with 16 * ((column / 8) % 4).  Aligned 16-element runs stay
// contiguous, so MFMA fragments (EL consecutive rows) remain 16-byte reads.
template <class P>
__device__ __forceinline__ int dw_swz(int col, int r) {
  if constexpr (P::EL == 4) return r;
  else return r ^ (16 * ((col >> 3) & 3));
}

// SPLIT (bf16 only): delta is fp32 and enters the products as hi + lo, two
// bf16 operands whose sum is within 2^-17 of it (relative).
template <int P_, bool SPLIT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2))) void dw_kernel(DwArgs a) {
  using P = typename PrecOf<P_>::type;
  using T = typename P::T;
  static_assert(!SPLIT || sizeof(T) == 2, "split operands are a bf16-mode form");
  constexpr int LDT = DW_RC + P::PAD;
  constexpr int GPR = DW_TO / P::EL;              // 16-byte groups per operand row
  constexpr int IT = DW_RC * GPR / NT;            // loads per thread per operand per chunk
  __shared__ __align__(16) T Dt[DW_TO * LDT];
  __shared__ __align__(16) T Dl[SPLIT ? DW_TO * LDT : 16];
  __shared__ __align__(16) T At[DW_TI * LDT];
  const int ot = blockIdx.x, itl = blockIdx.y, s = blockIdx.z;
  const int o0 = ot * DW_TO, i0 = itl * DW_TI;
  const int64_t per = (a.R + a.S - 1) / a.S;
  const int64_t rb = (int64_t)s * per, re = rb + per < a.R ? rb + per : a.R;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wo = (wave >> 1) * 64, wi = (wave & 1) * 64;  // this wave's 64x64 quadrant
  floatx4 acc[4][4];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};
  const T* dl = reinterpret_cast<const T*>(a.delta);
  // thread -> (row, column group): 16 consecutive rows per 16 lanes, four
  // column groups per wave (64 contiguous bytes of each row per wave)
  auto rowof = [&](int j) { const int idx = threadIdx.x + j * NT; return (idx & 15) + 16 * (idx / (16 * GPR)); };
  auto grpof = [&](int j) { const int idx = threadIdx.x + j * NT; return ((idx >> 4) % GPR) * P::EL; };
  uint4 rd[IT], ra[IT], rl[SPLIT ? IT : 1];
  auto load = [&](int64_t c0) {
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int r = rowof(j), g = grpof(j);
      const int64_t row = c0 + r;
      rd[j] = make_uint4(0, 0, 0, 0);
      ra[j] = make_uint4(0, 0, 0, 0);
      if constexpr (SPLIT) rl[j] = make_uint4(0, 0, 0, 0);
      if (row < re) {
        if constexpr (SPLIT) {
          // fp32 delta (a.O and a.ldd multiples of 8): 8 values, hi and lo halves
          if (o0 + g < a.O) {
            const float* src = reinterpret_cast<const float*>(a.delta) + row * a.ldd + o0 + g;
            const float4 x0 = reinterpret_cast<const float4*>(src)[0], x1 = reinterpret_cast<const float4*>(src)[1];
            const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
            uint16_t h[8], l[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              h[e] = f2bf(x[e]);
              l[e] = f2bf(x[e] - bf2f(h[e]));
            }
            rd[j] = *reinterpret_cast<const uint4*>(h);
            rl[j] = *reinterpret_cast<const uint4*>(l);
          }
        } else if (o0 + g < a.O) {
          if (o0 + g + P::EL <= a.ldd && (a.ldd % P::EL) == 0) {
            rd[j] = *reinterpret_cast<const uint4*>(dl + row * a.ldd + o0 + g);
          } else {
            T v[P::EL];
#pragma unroll
            for (int e = 0; e < P::EL; ++e) v[e] = (o0 + g + e < a.O) ? dl[row * a.ldd + o0 + g + e] : P::cvt(0.f);
            rd[j] = *reinterpret_cast<const uint4*>(v);
          }
        }
        if (i0 + g < a.I) ra[j] = dw_load_a<P>(a, row, i0 + g);
      }
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int r = rowof(j), g = grpof(j);
      const T* vd = reinterpret_cast<const T*>(&rd[j]);
      const T* va = reinterpret_cast<const T*>(&ra[j]);
#pragma unroll
      for (int e = 0; e < P::EL; ++e) {
        const int c = g + e;
        Dt[c * LDT + dw_swz<P>(c, r)] = (o0 + c < a.O) ? vd[e] : P::cvt(0.f);
        At[c * LDT + dw_swz<P>(c, r)] = (i0 + c < a.I) ? va[e] : P::cvt(0.f);
      }
      if constexpr (SPLIT) {
        const T* vl = reinterpret_cast<const T*>(&rl[j]);
#pragma unroll
        for (int e = 0; e < P::EL; ++e) {
          const int c = g + e;
          Dl[c * LDT + dw_swz<P>(c, r)] = (o0 + c < a.O) ? vl[e] : P::cvt(0.f);
        }
      }
    }
  };
  if (rb < re) load(rb);
  for (int64_t c0 = rb; c0 < re; c0 += DW_RC) {
    store();
    __syncthreads();
    if (c0 + DW_RC < re) load(c0 + DW_RC);  // next chunk in flight during the products
#pragma unroll
    for (int kg = 0; kg < DW_RC / P::KG; ++kg) {
      uint4 af[4], bf[4];
      const int kk = kg * P::KG + (lane >> 4) * P::EL;
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int c = wo + m * 16 + (lane & 15);
        af[m] = *reinterpret_cast<const uint4*>(Dt + c * LDT + dw_swz<P>(c, kk));
      }
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const int c = wi + n * 16 + (lane & 15);
        bf[n] = *reinterpret_cast<const uint4*>(At + c * LDT + dw_swz<P>(c, kk));
      }
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int n = 0; n < 4; ++n) P::mma(acc[m][n], af[m], bf[n]);
      if constexpr (SPLIT) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const int c = wo + m * 16 + (lane & 15);
          af[m] = *reinterpret_cast<const uint4*>(Dl + c * LDT + dw_swz<P>(c, kk));
        }
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
          for (int n = 0; n < 4; ++n) P::mma(acc[m][n], af[m], bf[n]);
      }
    }
    __syncthreads();
  }
  float* dst = a.part + (int64_t)s * a.O * a.I;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int n = 0; n < 4; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = o0 + wo + m * 16 + acc_row(r), i = i0 + wi + n * 16 + acc_col();
        if (o < a.O && i < a.I) dst[(int64_t)o * a.I + i] = acc[m][n][r];
      }
}

// ------------------------------------- weight gradients, register-resident ---
// dW = D^T A for bf16 row-major D [R][ldd] and A [R][lda], 128 columns each
// (the per-edge layers of the row-split path at l = 128), without LDS or
// barriers.  One wave per SIMD; each wave reduces a contiguous range of rows
// into a 128 x 128 fp32 tile held in the accumulator registers.  Per 32 rows,
// lane (q, m) = (lane >> 4, lane & 15) loads rows 8 q .. 8 q + 7, columns
// 8 m .. 8 m + 7 of both operands (16-byte loads: a wave instruction reads four
// whole rows), transposes each 8 x 8 block in registers into eight
// k-fragments (one column, eight consecutive rows) and issues 64 MFMAs:
// fragment j of lane (q, m) is column 8 m + j, so accumulator block (j, j')
// holds dW[8 m' + j][8 n + j'] at (row m', column n) of its 16 x 16 tile.
constexpr int DWS_NT = 256;
constexpr int DWS_GRID = 256;
constexpr int DWS_WAVES = DWS_GRID * DWS_NT / 64;

// v[r][k]: row r, columns 2k (low half) and 2k + 1 -> f[c][p]: column c, rows
// 2p (low half) and 2p + 1.
__device__ __forceinline__ void dws_transpose(const uint32_t (&v)[8][4], uint32_t (&f)[8][4]) {
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      f[2 * k][p] = __builtin_amdgcn_perm(v[2 * p + 1][k], v[2 * p][k], 0x05040100u);
      f[2 * k + 1][p] = __builtin_amdgcn_perm(v[2 * p + 1][k], v[2 * p][k], 0x07060302u);
    }
}

__device__ __forceinline__ void dws_load(const uint16_t* __restrict__ X, int ldx, int64_t row, int64_t R, int col,
                                         uint32_t (&v)[8][4]) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    uint4 t = make_uint4(0, 0, 0, 0);
    if (row + r < R) t = *reinterpret_cast<const uint4*>(X + (row + r) * ldx + col);
    v[r][0] = t.x;
    v[r][1] = t.y;
    v[r][2] = t.z;
    v[r][3] = t.w;
  }
}

// fp32 rows, rounded to bf16 (the products' operand) in the layout of dws_load.
__device__ __forceinline__ void dws_load_cvt(const float* __restrict__ X, int ldx, int64_t row, int64_t R, int col,
                                             uint32_t (&v)[8][4]) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
    if (row + r < R) {
      a = *reinterpret_cast<const float4*>(X + (row + r) * ldx + col);
      b = *reinterpret_cast<const float4*>(X + (row + r) * ldx + col + 4);
    }
    v[r][0] = (uint32_t)f2bf(a.x) | ((uint32_t)f2bf(a.y) << 16);
    v[r][1] = (uint32_t)f2bf(a.z) | ((uint32_t)f2bf(a.w) << 16);
    v[r][2] = (uint32_t)f2bf(b.x) | ((uint32_t)f2bf(b.y) << 16);
    v[r][3] = (uint32_t)f2bf(b.z) | ((uint32_t)f2bf(b.w) << 16);
  }
}

__device__ __forceinline__ void dws_mma(const uint32_t (&fd)[8][4], const uint32_t (&fa)[8][4], floatx4 (&acc)[8][8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj)
      PBF16::mma(acc[j][jj], make_uint4(fd[j][0], fd[j][1], fd[j][2], fd[j][3]),
                 make_uint4(fa[jj][0], fa[jj][1], fa[jj][2], fa[jj][3]));
}

// fp32 delta rows: 8 rows x 8 columns -> the bf16 hi and lo parts (x = hi +
// lo within 2^-17 relative), each as v[r][k] of dws_transpose.
__device__ __forceinline__ void dws_load_f32(const float* __restrict__ X, int ldx, int64_t row, int64_t R, int col,
                                             float4 (&v)[8][2]) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    v[r][0] = v[r][1] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (row + r < R) {
      v[r][0] = *reinterpret_cast<const float4*>(X + (row + r) * ldx + col);
      v[r][1] = *reinterpret_cast<const float4*>(X + (row + r) * ldx + col + 4);
    }
  }
}
__device__ __forceinline__ void dws_split(const float4 (&v)[8][2], uint32_t (&hi)[8][4], uint32_t (&lo)[8][4]) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const float x[8] = {v[r][0].x, v[r][0].y, v[r][0].z, v[r][0].w, v[r][1].x, v[r][1].y, v[r][1].z, v[r][1].w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint16_t h0 = f2bf(x[2 * k]), h1 = f2bf(x[2 * k + 1]);
      hi[r][k] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      lo[r][k] = (uint32_t)f2bf(x[2 * k] - bf2f(h0)) | ((uint32_t)f2bf(x[2 * k + 1] - bf2f(h1)) << 16);
    }
  }
}

// part[w] (16384 floats, accumulator order [j][j'][lane][4]) = wave w's sum.
// SPLIT: D is fp32 and enters the products as hi + lo (two MFMAs each).
// AF32: A is fp32, rounded to bf16 as it is loaded.
// QUAD: a 256 x 256 product.  The four waves of a workgroup take the same rows
// and one 128 x 128 quadrant each (wave v: D columns 128 (v >> 1) on, A
// columns 128 (v & 1) on), so each operand row is fetched from HBM once and
// its second reader finds it in the cache; part[v * gridDim.x + block] is
// quadrant v's partial of the workgroup's rows.
template <bool SPLIT, bool AF32 = false, bool QUAD = false>
__global__ __launch_bounds__(DWS_NT) __attribute__((amdgpu_waves_per_eu(1, 1))) void dw_stream_kernel(
    const void* __restrict__ Dv, int ldd, const void* __restrict__ Av, int lda, int64_t R,
    float* __restrict__ part) {
  const auto load_a = [&](int64_t row, int col, uint32_t (&v)[8][4]) {
    if constexpr (AF32)
      dws_load_cvt(reinterpret_cast<const float*>(Av), lda, row, R, col, v);
    else
      dws_load(reinterpret_cast<const uint16_t*>(Av), lda, row, R, col, v);
  };
  const int lane = threadIdx.x & 63, q = lane >> 4, m = lane & 15;
  const int wv = wave_id();
  const int64_t w = QUAD ? (int64_t)blockIdx.x : (int64_t)blockIdx.x * (DWS_NT / 64) + wv;
  const int64_t nw = QUAD ? (int64_t)gridDim.x : (int64_t)gridDim.x * (DWS_NT / 64);
  const int64_t steps = (R + 31) / 32;
  const int64_t s0 = steps * w / nw, s1 = steps * (w + 1) / nw;  // this wave's 32-row steps
  floatx4 acc[8][8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) acc[j][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int64_t rq = 8 * q;
  const int dc = (QUAD ? 128 * (wv >> 1) : 0) + 8 * m, ac = (QUAD ? 128 * (wv & 1) : 0) + 8 * m;
  // the next step's loads reuse the source registers once they are
  // transposed, so they are in flight during the current step's products
  if constexpr (SPLIT) {
    const float* D = reinterpret_cast<const float*>(Dv);
    float4 dv[8][2];
    uint32_t av[8][4], fa[8][4];
    if (s0 < s1) {
      dws_load_f32(D, ldd, s0 * 32 + rq, R, dc, dv);
      load_a(s0 * 32 + rq, ac, av);
    }
    for (int64_t st = s0; st < s1; ++st) {
      uint32_t hi[8][4], lo[8][4], f[8][4];
      dws_split(dv, hi, lo);
      dws_transpose(av, fa);
      if (st + 1 < s1) {
        dws_load_f32(D, ldd, (st + 1) * 32 + rq, R, dc, dv);
        load_a((st + 1) * 32 + rq, ac, av);
      }
      dws_transpose(hi, f);
      dws_mma(f, fa, acc);
      dws_transpose(lo, f);
      dws_mma(f, fa, acc);
    }
  } else {
    const uint16_t* D = reinterpret_cast<const uint16_t*>(Dv);
    uint32_t dv[8][4], av[8][4], fd[8][4], fa[8][4];
    if (s0 < s1) {
      dws_load(D, ldd, s0 * 32 + rq, R, dc, dv);
      load_a(s0 * 32 + rq, ac, av);
    }
    for (int64_t st = s0; st < s1; ++st) {
      dws_transpose(dv, fd);
      dws_transpose(av, fa);
      if (st + 1 < s1) {
        dws_load(D, ldd, (st + 1) * 32 + rq, R, dc, dv);
        load_a((st + 1) * 32 + rq, ac, av);
      }
      dws_mma(fd, fa, acc);
    }
  }
  float4* out =
      reinterpret_cast<float4*>(part + (QUAD ? (int64_t)wv * gridDim.x + blockIdx.x : w) * 16384);
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj)
      out[(j * 8 + jj) * 64 + lane] = make_float4(acc[j][jj][0], acc[j][jj][1], acc[j][jj][2], acc[j][jj][3]);
}

// fp32 form: dW = D^T A for fp32 row-major D [R][ldd] and A [R][lda], 128
// columns each (the per-edge layers at l = 128 in fp32).  The 16x16x4 fp32
// MFMA takes one value per lane, A[i][k] from lane (k, i) and B[k][j] from
// lane (k, j), so row-major loads need no transpose: per 4-row k-group, lane
// (q, m) = (lane >> 4, lane & 15) loads row q's columns 4m .. 4m + 3 and
// 64 + 4m .. 64 + 4m + 3 of both operands (float4 each), and component c of
// half h stands for column 64 h + 4 m + c; accumulator block (h, c, h', c')
// then holds dW[64 h + 4 i + c][64 h' + 4 j + c'] at (i, j) of its 16 x 16
// tile.  One wave per SIMD, 64 blocks = the 256 accumulator registers; a
// 16-row step's loads are issued one step ahead.  part[w] = wave w's sum in
// plain [o][i] order (reduced by dw_reduce_kernel).
__device__ __forceinline__ void dwf_load(const float* __restrict__ D, int ldd, const float* __restrict__ A, int lda,
                                         int64_t row, int64_t R, int m, float4 (&v)[4][4]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int64_t r = row + 4 * g;
    const bool ok = r < R;
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    v[g][0] = ok ? *reinterpret_cast<const float4*>(D + r * ldd + 4 * m) : z;
    v[g][1] = ok ? *reinterpret_cast<const float4*>(D + r * ldd + 64 + 4 * m) : z;
    v[g][2] = ok ? *reinterpret_cast<const float4*>(A + r * lda + 4 * m) : z;
    v[g][3] = ok ? *reinterpret_cast<const float4*>(A + r * lda + 64 + 4 * m) : z;
  }
}

__device__ __forceinline__ float f4c(const float4& v, int c) { return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w; }

__global__ __launch_bounds__(DWS_NT) __attribute__((amdgpu_waves_per_eu(1, 1))) void dw_stream_f32_kernel(
    const float* __restrict__ D, int ldd, const float* __restrict__ A, int lda, int64_t R, float* __restrict__ part) {
  const int lane = threadIdx.x & 63, q = lane >> 4, m = lane & 15;
  const int64_t w = (int64_t)blockIdx.x * (DWS_NT / 64) + wave_id();
  const int64_t nw = (int64_t)gridDim.x * (DWS_NT / 64);
  const int64_t steps = (R + 15) / 16;
  const int64_t s0 = steps * w / nw, s1 = steps * (w + 1) / nw;  // this wave's 16-row steps
  floatx4 acc[8][8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) acc[j][jj] = floatx4{0.f, 0.f, 0.f, 0.f};
  float4 cur[4][4], nxt[4][4];
  if (s0 < s1) dwf_load(D, ldd, A, lda, s0 * 16 + q, R, m, nxt);
  for (int64_t st = s0; st < s1; ++st) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int t = 0; t < 4; ++t) cur[g][t] = nxt[g][t];
    if (st + 1 < s1) dwf_load(D, ldd, A, lda, (st + 1) * 16 + q, R, m, nxt);
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int cc = 0; cc < 4; ++cc)
              acc[h * 4 + c][hh * 4 + cc] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  f4c(cur[g][h], c), f4c(cur[g][2 + hh], cc), acc[h * 4 + c][hh * 4 + cc], 0, 0, 0);
  }
  float* out = part + w * 16384;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int cc = 0; cc < 4; ++cc)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int o = 64 * h + 4 * (4 * q + r) + c, i = 64 * hh + 4 * m + cc;
            out[o * 128 + i] = acc[h * 4 + c][hh * 4 + cc][r];
          }
}

// dst[o * ldw + i] (+)= sum over the S wave partials, in wave order within
// each of four interleaved sets, combined in set order; entry x of a partial
// is (j, j', lane, r) -> o = 8 (4 (lane >> 4) + r) + j, i = 8 (lane & 15) + j'.
// gridDim.y > 1: quadrant y = blockIdx.y of a 256 x 256 gradient, its S
// partials from part + y S 16384, its outputs at rows 128 (y >> 1) and
// columns 128 (y & 1) on.
__global__ __launch_bounds__(NT) void dw_stream_reduce_kernel(const float* __restrict__ part, int S,
                                                              float* __restrict__ dst, int ldw, int accumulate) {
  __shared__ float sh[NT];
  const int jx = threadIdx.x & 63, qq = threadIdx.x >> 6;
  const int x = blockIdx.x * 64 + jx;
  part += (int64_t)blockIdx.y * S * 16384;
  dst += (int64_t)(blockIdx.y >> 1) * 128 * ldw + (blockIdx.y & 1) * 128;
  float t = 0.f;
#pragma unroll 8
  for (int k = qq; k < S; k += 4) t += part[(int64_t)k * 16384 + x];
  sh[threadIdx.x] = t;
  __syncthreads();
  if (qq == 0) {
    const float t4 = ((sh[jx] + sh[64 + jx]) + sh[128 + jx]) + sh[192 + jx];
    const int blk = x >> 8, ln = (x >> 2) & 63, r = x & 3;
    const int o = 8 * (4 * (ln >> 4) + r) + (blk >> 3), i = 8 * (ln & 15) + (blk & 7);
    float* d = dst + (int64_t)o * ldw + i;
    *d = (accumulate ? *d : 0.f) + t4;
  }
}

// dst[o * ldw + i] (+)= sum over the S split partials of part[.][o][i]: 64
// outputs per workgroup, four threads per output each summing the splits
// k = q (mod 4) in increasing k, combined in q order.
__global__ __launch_bounds__(NT) void dw_reduce_kernel(const float* __restrict__ part, int S, int O, int I,
                                                       float* __restrict__ dst, int ldw, int accumulate) {
  __shared__ float sh[NT];
  const int j = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t n = (int64_t)O * I;
  const int64_t i = (int64_t)blockIdx.x * 64 + j;
  float t = 0.f;
  if (i < n) {
#pragma unroll 8
    for (int k = q; k < S; k += 4) t += part[(int64_t)k * n + i];
  }
  sh[threadIdx.x] = t;
  __syncthreads();
  if (q == 0 && i < n) {
    const float t4 = ((sh[j] + sh[64 + j]) + sh[128 + j]) + sh[192 + j];
    float* d = dst + (i / I) * ldw + (i % I);
    const float s = accumulate ? *d : 0.f;
    *d = s + t4;
  }
}

struct VecSegs {
  VecSeg s[4];
  int n;
};

// The same four-way split of the slot sums as dw_reduce_kernel.
__global__ __launch_bounds__(NT) void vec_reduce_kernel(const float* __restrict__ vpart, int nwg, int nvec,
                                                        VecSegs segs, float* __restrict__ dparams, int accumulate) {
  __shared__ float sh[NT];
  const int j = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int i = blockIdx.x * 64 + j;
  float t = 0.f;
  if (i < nvec) {
#pragma unroll 8
    for (int w = q; w < nwg; w += 4) t += vpart[(int64_t)w * nvec + i];
  }
  sh[threadIdx.x] = t;
  __syncthreads();
  if (q != 0 || i >= nvec) return;
  t = ((sh[j] + sh[64 + j]) + sh[128 + j]) + sh[192 + j];
  for (int k = 0; k < segs.n; ++k) {
    const VecSeg& sg = segs.s[k];
    if (i >= sg.vec_off && i < sg.vec_off + sg.len) {
      float* d = dparams + sg.param_off + (i - sg.vec_off);
      *d = (accumulate ? *d : 0.f) + t;
    }
  }
}

// ------------------------------------------------------------------ loss ---
// Masked mean squared error: one workgroup sums count and squared error in a
// fixed order (double), then every element's gradient is written.
// Partial sums of the masked squared error, one per workgroup: (sum as fp64
// bits, selected row count) in 4 words at scratch + 4 * blockIdx.x.
constexpr int MSE_G = 256;
__global__ __launch_bounds__(NT) void mse_partial_kernel(const float* __restrict__ out, const float* __restrict__ tgt,
                                                         const uint8_t* __restrict__ mask, int64_t n, int d,
                                                         uint32_t* __restrict__ scratch) {
  __shared__ double ss[NT];
  __shared__ int64_t sc[NT];
  double s = 0.0;
  int64_t cnt = 0;
  for (int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x; i < n; i += (int64_t)gridDim.x * NT) {
    if (mask && !mask[i]) continue;
    ++cnt;
    for (int j = 0; j < d; ++j) {
      const double df = (double)out[i * d + j] - (double)tgt[i * d + j];
      s += df * df;
    }
  }
  ss[threadIdx.x] = s;
  sc[threadIdx.x] = cnt;
  __syncthreads();
  for (int w = NT / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      ss[threadIdx.x] += ss[threadIdx.x + w];
      sc[threadIdx.x] += sc[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const uint64_t b = __double_as_longlong(ss[0]);
    const uint64_t c = (uint64_t)sc[0];
    scratch[4 * blockIdx.x + 0] = (uint32_t)b;
    scratch[4 * blockIdx.x + 1] = (uint32_t)(b >> 32);
    scratch[4 * blockIdx.x + 2] = (uint32_t)c;
    scratch[4 * blockIdx.x + 3] = (uint32_t)(c >> 32);
  }
}

// Combines the MSE_G partials in workgroup order; writes the loss and the
// gradient scale 2 / (rows * d), rows = the masked row count, or grows when
// grows > 0 (a global mean over several parts: this part's share).
__global__ void mse_final_kernel(const uint32_t* __restrict__ scratch, int d, int64_t grows, float* __restrict__ loss,
                                 float* __restrict__ scale) {
  if (threadIdx.x != 0) return;
  double t = 0.0;
  int64_t c = 0;
  for (int b = 0; b < MSE_G; ++b) {
    const uint64_t bits = (uint64_t)scratch[4 * b] | ((uint64_t)scratch[4 * b + 1] << 32);
    t += __longlong_as_double((long long)bits);
    c += (int64_t)((uint64_t)scratch[4 * b + 2] | ((uint64_t)scratch[4 * b + 3] << 32));
  }
  if (grows > 0) c = grows;
  const double den = (double)c * d;
  *loss = c > 0 ? (float)(t / den) : 0.f;
  *scale = c > 0 ? (float)(2.0 / den) : 0.f;
}

__global__ __launch_bounds__(NT) void mse_loss_kernel(const float* __restrict__ out, const float* __restrict__ tgt,
                                                      const uint8_t* __restrict__ mask, int64_t n, int d,
                                                      int64_t grows, float* __restrict__ loss,
                                                      float* __restrict__ scale) {
  __shared__ double ss[NT];
  __shared__ int64_t sc[NT];
  double s = 0.0;
  int64_t cnt = 0;
  for (int64_t i = threadIdx.x; i < n; i += NT) {
    if (mask && !mask[i]) continue;
    ++cnt;
    for (int j = 0; j < d; ++j) {
      const double df = (double)out[i * d + j] - (double)tgt[i * d + j];
      s += df * df;
    }
  }
  ss[threadIdx.x] = s;
  sc[threadIdx.x] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    int64_t c = 0;
    for (int i = 0; i < NT; ++i) {
      t += ss[i];
      c += sc[i];
    }
    if (grows > 0) c = grows;
    const double den = (double)c * d;
    *loss = c > 0 ? (float)(t / den) : 0.f;
    *scale = c > 0 ? (float)(2.0 / den) : 0.f;
  }
}

__global__ void mse_grad_kernel(const float* __restrict__ out, const float* __restrict__ tgt,
                                const uint8_t* __restrict__ mask, int64_t n, int d, const float* __restrict__ scale,
                                float* __restrict__ d_out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n * d) return;
  const int64_t row = i / d;
  const bool on = mask ? mask[row] != 0 : true;
  d_out[i] = on ? (out[i] - tgt[i]) * *scale : 0.f;
}

// ============================================================ launchers ===
int edge_tile_rows(int prec, int L, int D) {
#define ETR(PP, LL, DD) \
  if (prec == PP && L == LL && D == DD) return EdgeTE<typename PrecOf<PP>::type, LL, DD>::value;
  ETR(F32, 64, 2) ETR(F32, 64, 3) ETR(F32, 128, 2) ETR(F32, 128, 3) ETR(F32, 256, 2) ETR(F32, 256, 3)
  ETR(BF16, 64, 2) ETR(BF16, 64, 3) ETR(BF16, 128, 2) ETR(BF16, 128, 3) ETR(BF16, 256, 2) ETR(BF16, 256, 3)
#undef ETR
  return 0;
}

hipError_t launch_pack(int prec, const float* W, int out, int in, int bwd, uint4* dst, int nkg, hipStream_t st) {
  const int nblk = ((bwd ? in : out) + 15) / 16;
  const int64_t total = (int64_t)nblk * nkg * 64;
  const int grid = (int)((total + NT - 1) / NT);
  if (prec == F32)
    hipLaunchKernelGGL(pack_kernel<PF32>, dim3(grid), dim3(NT), 0, st, W, out, in, bwd, dst, nkg, total);
  else
    hipLaunchKernelGGL(pack_kernel<PBF16>, dim3(grid), dim3(NT), 0, st, W, out, in, bwd, dst, nkg, total);
  return hipGetLastError();
}

hipError_t launch_erecv(const int32_t* row_ptr, int64_t n_owned, int32_t* erecv, hipStream_t st) {
  if (n_owned == 0) return hipSuccess;
  hipLaunchKernelGGL(erecv_kernel, dim3((unsigned)((n_owned + NT - 1) / NT)), dim3(NT), 0, st, row_ptr, n_owned,
                     erecv);
  return hipGetLastError();
}

int64_t plan_chunks(int64_t n_owned) { return (n_owned + PLAN_CHUNK - 1) / PLAN_CHUNK; }
int plan_chunk_receivers() { return PLAN_CHUNK; }

int64_t plan_max_units(int64_t n_owned, int64_t n_edges, int te_target, int r_max) {
  // a closed unit plus the receiver that closed it exceeds te_target edges or
  // r_max receivers, so two consecutive units hold more than min(te_target,
  // r_max) of edges+receivers; each chunk adds at most one partial unit.
  const int64_t lim = te_target < r_max ? te_target : r_max;
  return 2 * (n_owned + n_edges) / lim + 2 * plan_chunks(n_owned) + 2;
}

hipError_t launch_plan(const int32_t* row_ptr, int64_t n_owned, int te_target, int r_max, int32_t* chunk_cnt,
                       int32_t* unit_r, int32_t* n_units, hipStream_t st) {
  const int64_t nch = plan_chunks(n_owned);
  if (nch == 0) {
    // no receivers: zero units, unit_r[0] = 0
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, st, n_units, (int64_t)1, 0);
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, st, unit_r, (int64_t)1, 0);
    return hipGetLastError();
  }
  const unsigned g = (unsigned)((nch + NT - 1) / NT);
  hipLaunchKernelGGL(plan_count_kernel, dim3(g), dim3(NT), 0, st, row_ptr, n_owned, te_target, r_max, chunk_cnt,
                     nch);
  hipLaunchKernelGGL(plan_scan_kernel, dim3(1), dim3(NT), 0, st, chunk_cnt, nch, n_units);
  hipLaunchKernelGGL(plan_write_kernel, dim3(g), dim3(NT), 0, st, row_ptr, n_owned, te_target, r_max, chunk_cnt,
                     nch, n_units, unit_r);
  return hipGetLastError();
}

// Dynamic LDS above 64 KiB must be allowed explicitly per kernel.
template <class F>
static void allow_lds(F* fn, int bytes) {
  if (bytes > 65536) (void)hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

template <int P_, int L, int D, int KIND>
static hipError_t rows_fwd_t(const RowsFwdArgs& a, hipStream_t st) {
  using P = typename PrecOf<P_>::type;
  constexpr int TM = RowTM<P, KIND, L, D>::value;
  using Lay = RowLds<P, KIND, L, D, TM>;
  const int64_t ntiles = (a.rows + TM - 1) / TM;
  if (ntiles == 0) return hipSuccess;
  const int grid = (int)(ntiles < 4096 ? ntiles : 4096);
  allow_lds(rows_fwd_kernel<P_, L, D, KIND>, Lay::END_F);
  hipLaunchKernelGGL((rows_fwd_kernel<P_, L, D, KIND>), dim3(grid), dim3(NT), Lay::END_F, st, a);
  return hipGetLastError();
}

template <int P_, int L, int D, int KIND>
static hipError_t rows_bwd_t(const RowsBwdArgs& a, int grid, hipStream_t st) {
  using P = typename PrecOf<P_>::type;
  constexpr int TM = RowTM<P, KIND, L, D>::value;
  using Lay = RowLds<P, KIND, L, D, TM>;
  allow_lds(rows_bwd_kernel<P_, L, D, KIND>, Lay::END_B);
  hipLaunchKernelGGL((rows_bwd_kernel<P_, L, D, KIND>), dim3(grid), dim3(NT), Lay::END_B, st, a);
  return hipGetLastError();
}

template <int P_, int L, int D>
static hipError_t edge_fwd_t(const EdgeFwdArgs& a, int grid, hipStream_t st) {
  using P = typename PrecOf<P_>::type;
  using Lay = EdgeLds<P, L, D, EdgeTE<P, L, D>::value>;
  allow_lds(edge_fwd_kernel<P_, L, D>, Lay::END_F);
  hipLaunchKernelGGL((edge_fwd_kernel<P_, L, D>), dim3(grid), dim3(NT), Lay::END_F, st, a);
  return hipGetLastError();
}

template <int P_, int L, int D>
static hipError_t edge_bwd_t(const EdgeBwdArgs& a, int grid, hipStream_t st) {
  using P = typename PrecOf<P_>::type;
  using Lay = EdgeBwdLds<P, L, D, EdgeTEB<P, L, D>::value>;
  // the way h_1 is obtained: the forward's copy or the gathered rows
  if (a.hid_in) {
    allow_lds(edge_bwd_kernel<P_, L, D, BWD_STASH>, Lay::END);
    hipLaunchKernelGGL((edge_bwd_kernel<P_, L, D, BWD_STASH>), dim3(grid), dim3(NT), Lay::END, st, a);
  } else {
    allow_lds(edge_bwd_kernel<P_, L, D, BWD_GATHER>, Lay::END);
    hipLaunchKernelGGL((edge_bwd_kernel<P_, L, D, BWD_GATHER>), dim3(grid), dim3(NT), Lay::END, st, a);
  }
  return hipGetLastError();
}

bool rows_rt(int prec, int L, int D, int kind) {
  return prec == BF16 && D == 2 && (L == 64 || L == 128) && kind != DECODER;
}

bool rows_rw(int prec, int L, int D, int kind) {
  return prec == BF16 && L == 256 && (D == 2 || D == 3) && (kind == NODE_BLOCK || kind == ENC_EDGE);
}

bool rows_keep_h1(int prec, int L, int D) { return rows_rt(prec, L, D, NODE_BLOCK) || rows_rw(prec, L, D, NODE_BLOCK); }

template <int D>
static hipError_t rows_rw_fwd_t(const RowsFwdArgs& a, hipStream_t st) {
  using Lay = RwNodeFwdLay<D>;
  if (a.rows == 0) return hipSuccess;
  if (!a.in0_16 || !a.in1 || (a.out && !a.in0)) return hipErrorInvalidValue;
  allow_lds(rows_rw_fwd_kernel<D>, Lay::END);
  hipLaunchKernelGGL((rows_rw_fwd_kernel<D>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

template <int D>
static hipError_t rows_rw_enc_fwd_t(const RowsFwdArgs& a, hipStream_t st) {
  using Lay = RwEncFwdLay<D>;
  if (a.rows == 0) return hipSuccess;
  if (!a.in0 || !a.out || a.fin < 1 || a.fin > RW_ENC_FIN) return hipErrorInvalidValue;
  allow_lds(rows_rw_enc_fwd_kernel<D>, Lay::END);
  hipLaunchKernelGGL((rows_rw_enc_fwd_kernel<D>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

template <int D>
static hipError_t rows_rw_enc_bwd_t(const RowsBwdArgs& a, hipStream_t st) {
  using Lay = RwEncBwdLay<D>;
  if (!a.in0 || a.fin < 1 || a.fin > RW_ENC_FIN || a.nvec != Lay::NVEC) return hipErrorInvalidValue;
  allow_lds(rows_rw_enc_bwd_kernel<D>, Lay::END);
  hipLaunchKernelGGL((rows_rw_enc_bwd_kernel<D>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

template <int D>
static hipError_t rows_rw_bwd_t(const RowsBwdArgs& a, hipStream_t st) {
  using Lay = RwNodeBwdLay<D>;
  if (!a.hid_in || a.nvec != Lay::NVEC) return hipErrorInvalidValue;
  allow_lds(rows_rw_bwd_kernel<D>, Lay::END);
  hipLaunchKernelGGL((rows_rw_bwd_kernel<D>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

template <int L, int KIND>
static hipError_t rows_rt_fwd_t(const RowsFwdArgs& a, hipStream_t st) {
  using Lay = RtRowsLay<L, KIND>;
  if (a.rows == 0) return hipSuccess;
  allow_lds(rows_rt_fwd_kernel<L, KIND>, Lay::F_END);
  hipLaunchKernelGGL((rows_rt_fwd_kernel<L, KIND>), dim3(RS_GRID), dim3(Lay::FNTH), Lay::F_END, st, a);
  return hipGetLastError();
}

template <int L, int KIND>
static hipError_t rows_rt_bwd_t(const RowsBwdArgs& a, hipStream_t st) {
  using Lay = RtRowsLay<L, KIND>;
  if (a.w1_part && (KIND != ENC_EDGE || a.fin > Lay::W1_FIN || a.fin < 1)) return hipErrorInvalidValue;
  const int lds = a.w1_part ? Lay::B_END_W1 : Lay::B_END;
  allow_lds(rows_rt_bwd_kernel<L, KIND>, Lay::B_END_W1);
  hipLaunchKernelGGL((rows_rt_bwd_kernel<L, KIND>), dim3(RS_GRID), dim3(Lay::NTH), lds, st, a);
  return hipGetLastError();
}

// the partials fit the weight-gradient partial buffer, which holds at least
// the register-resident kernel's DWS_WAVES x 16384 floats
static_assert((int64_t)RS_GRID * RtRowsLay<128, ENC_EDGE>::NWV * 128 * RtRowsLay<128, ENC_EDGE>::W1_FIN <=
                  (int64_t)DWS_WAVES * 16384,
              "w1 partials");
int rows_rt_w1_parts(int prec, int L, int D, int kind, int fin) {
  if (kind != ENC_EDGE || fin < 1) return 0;
  if (rows_rw(prec, L, D, kind)) return fin <= RW_ENC_FIN ? RS_GRID * RwEncBwdLay<3>::NWV : 0;
  if (!rows_rt(prec, L, D, kind) || fin > RtRowsLay<128, ENC_EDGE>::W1_FIN) return 0;
  return RS_GRID * RtRowsLay<128, ENC_EDGE>::NWV;
}

hipError_t launch_rows_fwd(int prec, int L, int D, int kind, const RowsFwdArgs& a, hipStream_t st) {
  if (rows_rw(prec, L, D, kind)) {
    if (kind == ENC_EDGE) return D == 2 ? rows_rw_enc_fwd_t<2>(a, st) : rows_rw_enc_fwd_t<3>(a, st);
    return D == 2 ? rows_rw_fwd_t<2>(a, st) : rows_rw_fwd_t<3>(a, st);
  }
  if (rows_rt(prec, L, D, kind)) {
    if (L == 64) {
      if (kind == ENC_NODE) return rows_rt_fwd_t<64, ENC_NODE>(a, st);
      if (kind == ENC_EDGE) return rows_rt_fwd_t<64, ENC_EDGE>(a, st);
      return rows_rt_fwd_t<64, NODE_BLOCK>(a, st);
    }
    if (kind == ENC_NODE) return rows_rt_fwd_t<128, ENC_NODE>(a, st);
    if (kind == ENC_EDGE) return rows_rt_fwd_t<128, ENC_EDGE>(a, st);
    return rows_rt_fwd_t<128, NODE_BLOCK>(a, st);
  }
#define RF(PP, LL, DD)                                                                      \
  if (prec == PP && L == LL && D == DD) {                                                   \
    switch (kind) {                                                                         \
      case ENC_NODE: return rows_fwd_t<PP, LL, DD, ENC_NODE>(a, st);                        \
      case ENC_EDGE: return rows_fwd_t<PP, LL, DD, ENC_EDGE>(a, st);                        \
      case NODE_BLOCK: return rows_fwd_t<PP, LL, DD, NODE_BLOCK>(a, st);                    \
      default: return rows_fwd_t<PP, LL, DD, DECODER>(a, st);                               \
    }                                                                                       \
  }
  RF(F32, 64, 2) RF(F32, 64, 3) RF(F32, 128, 2) RF(F32, 128, 3) RF(F32, 256, 2) RF(F32, 256, 3)
  RF(BF16, 64, 2) RF(BF16, 64, 3) RF(BF16, 128, 2) RF(BF16, 128, 3) RF(BF16, 256, 2) RF(BF16, 256, 3)
#undef RF
  return hipErrorInvalidValue;
}

static bool rows_rs(int prec, int L, int D, int kind) {
  return prec == BF16 && D == 2 && (L == 64 || L == 128) && (kind == NODE_BLOCK || kind == ENC_EDGE);
}

// Backward kinds on the T-form kernel (NODE_BLOCK only with the forward's
// ReLU output at hand).
static bool rows_rt_bwd(int prec, int L, int D, int kind, bool hid_in) {
  return rows_rt(prec, L, D, kind) && (kind == ENC_EDGE || kind == ENC_NODE || (kind == NODE_BLOCK && hid_in));
}

int rows_bwd_grid(int prec, int L, int D, int kind, int grid) {
  return rows_rs(prec, L, D, kind) || rows_rt_bwd(prec, L, D, kind, false) || rows_rw(prec, L, D, kind) ? RS_GRID
                                                                                                       : grid;
}

template <int L, int KIND>
static hipError_t rows_bwd_rs_t(const RowsBwdArgs& a, hipStream_t st) {
  using Lay = RsRowsLay<L, KIND>;
  allow_lds(rows_bwd_rs_kernel<L, KIND>, Lay::END);
  hipLaunchKernelGGL((rows_bwd_rs_kernel<L, KIND>), dim3(RS_GRID), dim3(RS_NTH), Lay::END, st, a);
  return hipGetLastError();
}

hipError_t launch_rows_bwd(int prec, int L, int D, int kind, const RowsBwdArgs& a, int grid, hipStream_t st) {
  if (rows_rw(prec, L, D, kind)) {
    if (kind == ENC_EDGE) return D == 2 ? rows_rw_enc_bwd_t<2>(a, st) : rows_rw_enc_bwd_t<3>(a, st);
    return D == 2 ? rows_rw_bwd_t<2>(a, st) : rows_rw_bwd_t<3>(a, st);
  }
  if (rows_rt_bwd(prec, L, D, kind, a.hid_in != nullptr)) {
    if (L == 64) {
      if (kind == ENC_NODE) return rows_rt_bwd_t<64, ENC_NODE>(a, st);
      return kind == ENC_EDGE ? rows_rt_bwd_t<64, ENC_EDGE>(a, st) : rows_rt_bwd_t<64, NODE_BLOCK>(a, st);
    }
    if (kind == ENC_NODE) return rows_rt_bwd_t<128, ENC_NODE>(a, st);
    return kind == ENC_EDGE ? rows_rt_bwd_t<128, ENC_EDGE>(a, st) : rows_rt_bwd_t<128, NODE_BLOCK>(a, st);
  }
  if (rows_rs(prec, L, D, kind)) {
    if (L == 64) return kind == NODE_BLOCK ? rows_bwd_rs_t<64, NODE_BLOCK>(a, st) : rows_bwd_rs_t<64, ENC_EDGE>(a, st);
    return kind == NODE_BLOCK ? rows_bwd_rs_t<128, NODE_BLOCK>(a, st) : rows_bwd_rs_t<128, ENC_EDGE>(a, st);
  }
#define RB(PP, LL, DD)                                                                      \
  if (prec == PP && L == LL && D == DD) {                                                   \
    switch (kind) {                                                                         \
      case ENC_NODE: return rows_bwd_t<PP, LL, DD, ENC_NODE>(a, grid, st);                  \
      case ENC_EDGE: return rows_bwd_t<PP, LL, DD, ENC_EDGE>(a, grid, st);                  \
      case NODE_BLOCK: return rows_bwd_t<PP, LL, DD, NODE_BLOCK>(a, grid, st);              \
      default: return rows_bwd_t<PP, LL, DD, DECODER>(a, grid, st);                         \
    }                                                                                       \
  }
  RB(F32, 64, 2) RB(F32, 64, 3) RB(F32, 128, 2) RB(F32, 128, 3) RB(F32, 256, 2) RB(F32, 256, 3)
  RB(BF16, 64, 2) RB(BF16, 64, 3) RB(BF16, 128, 2) RB(BF16, 128, 3) RB(BF16, 256, 2) RB(BF16, 256, 3)
#undef RB
  return hipErrorInvalidValue;
}

bool edge_rs(int prec, int L, int D) { return prec == BF16 && (L == 64 || (L == 128 && D == 2)); }

template <int L, int D>
static hipError_t edge_fwd_rs_t(const EdgeFwdArgs& a, hipStream_t st) {
  using Lay = RsFwdLay<L, D>;
  allow_lds(edge_fwd_rs_kernel<L, D>, Lay::END);
  hipLaunchKernelGGL((edge_fwd_rs_kernel<L, D>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

template <int L, int D>
static hipError_t edge_bwd_rs_t(const EdgeBwdArgs& a, hipStream_t st) {
  using Lay = RsBwdLay<L, D>;
  if (a.hid_in) {
    allow_lds(edge_bwd_rs_kernel<L, D, true>, Lay::END);
    hipLaunchKernelGGL((edge_bwd_rs_kernel<L, D, true>), dim3(RS_GRID), dim3(RS_NTH), Lay::END, st, a);
  } else {
    allow_lds(edge_bwd_rs_kernel<L, D, false>, Lay::END);
    hipLaunchKernelGGL((edge_bwd_rs_kernel<L, D, false>), dim3(RS_GRID), dim3(RS_NTH), Lay::END, st, a);
  }
  return hipGetLastError();
}

template <int L>
static hipError_t node_proj_t(const void* v16, int64_t n_local, const Lin& w1, float* proj, hipStream_t st) {
  constexpr int W = (L / 16) * (L / 32) * 64 * 16;
  allow_lds(node_proj_kernel<L>, 2 * W);
  hipLaunchKernelGGL((node_proj_kernel<L>), dim3(RS_GRID), dim3(RS_NTH), 2 * W, st,
                     reinterpret_cast<const uint16_t*>(v16), n_local, w1, proj);
  return hipGetLastError();
}

hipError_t launch_node_proj(int L, const void* v16, int64_t n_local, const Lin& w1, float* proj, hipStream_t st) {
  if (n_local == 0) return hipSuccess;
  if (L == 64) return node_proj_t<64>(v16, n_local, w1, proj, st);
  if (L == 128) return node_proj_t<128>(v16, n_local, w1, proj, st);
  if (L == 256) {
    allow_lds(node_proj_rw_kernel, RwProjLay::END);
    hipLaunchKernelGGL(node_proj_rw_kernel, dim3(RS_GRID), dim3(RwProjLay::NTH), RwProjLay::END, st,
                       reinterpret_cast<const uint16_t*>(v16), n_local, w1, proj);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

bool edge_rsb(int prec, int L, int D) { return prec == BF16 && L == 256 && (D == 2 || D == 3); }


template <int D, int NS, int NWV>
static hipError_t edge_fwd_rw_t(const EdgeFwdArgs& a, hipStream_t st) {
  using Lay = RwFwdLay<D, NS, NWV>;
  allow_lds(edge_fwd_rw_kernel<D, NS, NWV>, Lay::END);
  hipLaunchKernelGGL((edge_fwd_rw_kernel<D, NS, NWV>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

// the l = 256 forward's tile shape: edges per wave (16 x RW_FWD_NS) and waves
// per workgroup
#ifndef RW_FWD_NS
#define RW_FWD_NS 1
#endif
#ifndef RW_FWD_NWV
#define RW_FWD_NWV 8
#endif

hipError_t launch_edge_fwd(int prec, int L, int D, const EdgeFwdArgs& a, int grid, hipStream_t st) {
  if (edge_rsb(prec, L, D)) {
    if (!a.proj) return hipErrorInvalidValue;
    return D == 2 ? edge_fwd_rw_t<2, RW_FWD_NS, RW_FWD_NWV>(a, st) : edge_fwd_rw_t<3, RW_FWD_NS, RW_FWD_NWV>(a, st);
  }
  if (edge_rs(prec, L, D)) {
    if (L == 64) return D == 2 ? edge_fwd_rs_t<64, 2>(a, st) : edge_fwd_rs_t<64, 3>(a, st);
    return edge_fwd_rs_t<128, 2>(a, st);
  }
#define EF(PP, LL, DD) \
  if (prec == PP && L == LL && D == DD) return edge_fwd_t<PP, LL, DD>(a, grid, st);
  EF(F32, 64, 2) EF(F32, 64, 3) EF(F32, 128, 2) EF(F32, 128, 3) EF(F32, 256, 2) EF(F32, 256, 3)
  EF(BF16, 64, 2) EF(BF16, 64, 3) EF(BF16, 128, 2) EF(BF16, 128, 3) EF(BF16, 256, 2) EF(BF16, 256, 3)
#undef EF
  return hipErrorInvalidValue;
}

int edge_bwd_grid(int prec, int L, int D, int grid) {
  return edge_rs(prec, L, D) || edge_rsb(prec, L, D) ? RS_GRID : grid;
}

#ifndef RW_BWD_NWV
#define RW_BWD_NWV 4
#endif

template <int D, bool STASH>
static hipError_t edge_bwd_rw_t(const EdgeBwdArgs& a, hipStream_t st) {
  using Lay = RwBwdLay<D, STASH, RW_BWD_NWV>;
  allow_lds(edge_bwd_rw_kernel<D, STASH, RW_BWD_NWV>, Lay::END);
  hipLaunchKernelGGL((edge_bwd_rw_kernel<D, STASH, RW_BWD_NWV>), dim3(RS_GRID), dim3(Lay::NTH), Lay::END, st, a);
  return hipGetLastError();
}

hipError_t launch_edge_bwd(int prec, int L, int D, const EdgeBwdArgs& a, int grid, hipStream_t st) {
  if (edge_rsb(prec, L, D)) {
    // h_1 from the forward's copy, or recomputed from e and the projections
    if (a.hid_in) return D == 2 ? edge_bwd_rw_t<2, true>(a, st) : edge_bwd_rw_t<3, true>(a, st);
    if (!a.proj) return hipErrorInvalidValue;
    return D == 2 ? edge_bwd_rw_t<2, false>(a, st) : edge_bwd_rw_t<3, false>(a, st);
  }
  if (edge_rs(prec, L, D)) {
    if (L == 64) return D == 2 ? edge_bwd_rs_t<64, 2>(a, st) : edge_bwd_rs_t<64, 3>(a, st);
    return edge_bwd_rs_t<128, 2>(a, st);
  }
#define EB(PP, LL, DD) \
  if (prec == PP && L == LL && D == DD) return edge_bwd_t<PP, LL, DD>(a, grid, st);
  EB(F32, 64, 2) EB(F32, 64, 3) EB(F32, 128, 2) EB(F32, 128, 3) EB(F32, 256, 2) EB(F32, 256, 3)
  EB(BF16, 64, 2) EB(BF16, 64, 3) EB(BF16, 128, 2) EB(BF16, 128, 3) EB(BF16, 256, 2) EB(BF16, 256, 3)
#undef EB
  return hipErrorInvalidValue;
}

template <int P_, int L>
static hipError_t input_grad_t(const InGradArgs& a, hipStream_t st) {
  using P = typename PrecOf<P_>::type;
  using G = InGradTile<P, L>;
  allow_lds(input_grad_kernel<P_, L>, G::END);
  const unsigned grid = (unsigned)((a.n_local + G::TM - 1) / G::TM);
  hipLaunchKernelGGL((input_grad_kernel<P_, L>), dim3(grid), dim3(NT), G::END, st, a);
  return hipGetLastError();
}

template <int P_, int L>
static hipError_t sender_sums_t(const int32_t* trow, const int32_t* tedge, const void* dz, int64_t e_lo, int64_t e_hi,
                                int64_t n_local, float* dzs, int first, const int32_t* range, hipStream_t st) {
  constexpr int CPR = L / (16 / (P_ == BF16 ? 2 : 4));
  int64_t grid = (n_local * CPR + NT - 1) / NT;
  if (range && grid > 4096) grid = 4096;  // a grid-stride loop over the range read on the device
  hipLaunchKernelGGL((sender_sums_kernel<P_, L>), dim3((unsigned)grid), dim3(NT), 0, st, trow, tedge, dz, e_lo, e_hi,
                     n_local, dzs, first, range);
  return hipGetLastError();
}

hipError_t launch_sender_sums(int prec, int L, const int32_t* trow, const int32_t* tedge, const void* dz, int64_t e_lo,
                              int64_t e_hi, int64_t n_local, float* dzs, int first, const int32_t* range,
                              hipStream_t st) {
  if (n_local == 0) return hipSuccess;
#define SS(PP, LL) \
  if (prec == PP && L == LL) return sender_sums_t<PP, LL>(trow, tedge, dz, e_lo, e_hi, n_local, dzs, first, range, st);
  SS(F32, 64) SS(F32, 128) SS(F32, 256) SS(BF16, 64) SS(BF16, 128) SS(BF16, 256)
#undef SS
  return hipErrorInvalidValue;
}

hipError_t launch_sender_range(const int32_t* send, int64_t e_lo, int64_t e_hi, int32_t* range, hipStream_t st) {
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, st, range, (int64_t)1, (int32_t)INT32_MAX);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(64), 0, st, range + 1, (int64_t)1, (int32_t)-1);
  const int64_t n = e_hi - e_lo;
  if (n > 0) {
    int64_t grid = (n + NT - 1) / NT;
    if (grid > 1024) grid = 1024;
    hipLaunchKernelGGL(sender_range_kernel, dim3((unsigned)grid), dim3(NT), 0, st, send, e_lo, e_hi, range);
  }
  return hipGetLastError();
}

hipError_t launch_input_grad(int prec, int L, const InGradArgs& a, hipStream_t st) {
  if (a.n_local == 0) return hipSuccess;
#define IG(PP, LL) \
  if (prec == PP && L == LL) return input_grad_t<PP, LL>(a, st);
  IG(F32, 64) IG(F32, 128) IG(F32, 256) IG(BF16, 64) IG(BF16, 128) IG(BF16, 256)
#undef IG
  return hipErrorInvalidValue;
}

int dw_splits(int64_t R, int O, int I) {
  const int64_t tiles = (int64_t)((O + DW_TO - 1) / DW_TO) * ((I + DW_TI - 1) / DW_TI);
  int64_t s = 2048 / tiles;
  const int64_t by_rows = (R + 4 * DW_RC - 1) / (4 * DW_RC);  // at least 4 chunks per split
  if (s > by_rows) s = by_rows;
  if (s < 1) s = 1;
  return (int)s;
}

hipError_t launch_dw(int prec, const DwArgs& a, hipStream_t st) {
  dim3 grid((a.O + DW_TO - 1) / DW_TO, (a.I + DW_TI - 1) / DW_TI, a.S);
  if (a.d_kind == 1 && (a.O % 8 != 0 || a.ldd % 8 != 0)) return hipErrorInvalidValue;
  if (prec == F32)
    hipLaunchKernelGGL((dw_kernel<F32, false>), grid, dim3(NT), 0, st, a);
  else if (a.d_kind == 1)
    hipLaunchKernelGGL((dw_kernel<BF16, true>), grid, dim3(NT), 0, st, a);
  else
    hipLaunchKernelGGL((dw_kernel<BF16, false>), grid, dim3(NT), 0, st, a);
  return hipGetLastError();
}

int dw_stream_parts() { return DWS_WAVES; }

bool dw_stream_f32_ok(int prec, const DwArgs& a) {
  return prec == F32 && a.a_kind == 0 && a.d_kind == 0 && a.O == 128 && a.I == 128 && a.ldd % 4 == 0 &&
         a.lda0 % 4 == 0 && a.R >= 8192 && ((uintptr_t)a.delta % 16) == 0 && ((uintptr_t)a.a0 % 16) == 0;
}

hipError_t launch_dw_stream_f32(const DwArgs& a, float* dst, int ldw, int accumulate, hipStream_t st) {
  hipLaunchKernelGGL(dw_stream_f32_kernel, dim3(DWS_GRID), dim3(DWS_NT), 0, st,
                     reinterpret_cast<const float*>(a.delta), a.ldd, reinterpret_cast<const float*>(a.a0), a.lda0,
                     a.R, a.part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_dw_reduce(a.part, DWS_WAVES, 128, 128, dst, ldw, accumulate, st);
}

bool dw_stream_ok(int prec, const DwArgs& a) {
  // A: bf16 rows (a_kind 0) or fp32 rows rounded on load (a_kind 1, bf16 delta)
  return prec == BF16 && (a.a_kind == 0 || (a.a_kind == 1 && a.d_kind == 0)) &&
         (a.d_kind == 0 || a.d_kind == 1) && a.O == 128 && a.I == 128 && a.ldd % 8 == 0 && a.lda0 % 8 == 0 &&
         a.R >= 8192;
}

hipError_t launch_dw_stream(const DwArgs& a, float* dst, int ldw, int accumulate, hipStream_t st) {
  if (a.d_kind == 1)
    hipLaunchKernelGGL((dw_stream_kernel<true, false>), dim3(DWS_GRID), dim3(DWS_NT), 0, st, a.delta, a.ldd, a.a0,
                       a.lda0, a.R, a.part);
  else if (a.a_kind == 1)
    hipLaunchKernelGGL((dw_stream_kernel<false, true>), dim3(DWS_GRID), dim3(DWS_NT), 0, st, a.delta, a.ldd, a.a0,
                       a.lda0, a.R, a.part);
  else
    hipLaunchKernelGGL((dw_stream_kernel<false, false>), dim3(DWS_GRID), dim3(DWS_NT), 0, st, a.delta, a.ldd, a.a0,
                       a.lda0, a.R, a.part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(dw_stream_reduce_kernel, dim3(16384 / 64), dim3(NT), 0, st, a.part, DWS_WAVES, dst, ldw,
                     accumulate);
  return hipGetLastError();
}

bool dw_stream_quad_ok(int prec, const DwArgs& a) {
  return prec == BF16 && (a.a_kind == 0 || (a.a_kind == 1 && a.d_kind == 0)) &&
         (a.d_kind == 0 || a.d_kind == 1) && a.O == 256 && a.I == 256 && a.ldd % 8 == 0 && a.lda0 % 8 == 0 &&
         a.R >= 8192;
}

hipError_t launch_dw_stream_quad(const DwArgs& a, float* dst, int ldw, int accumulate, hipStream_t st) {
  // DWS_GRID workgroups x 4 quadrants = the DWS_WAVES partials of the plain form
  if (a.d_kind == 1)
    hipLaunchKernelGGL((dw_stream_kernel<true, false, true>), dim3(DWS_GRID), dim3(DWS_NT), 0, st, a.delta, a.ldd,
                       a.a0, a.lda0, a.R, a.part);
  else if (a.a_kind == 1)
    hipLaunchKernelGGL((dw_stream_kernel<false, true, true>), dim3(DWS_GRID), dim3(DWS_NT), 0, st, a.delta, a.ldd,
                       a.a0, a.lda0, a.R, a.part);
  else
    hipLaunchKernelGGL((dw_stream_kernel<false, false, true>), dim3(DWS_GRID), dim3(DWS_NT), 0, st, a.delta, a.ldd,
                       a.a0, a.lda0, a.R, a.part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(dw_stream_reduce_kernel, dim3(16384 / 64, 4), dim3(NT), 0, st, a.part, DWS_GRID, dst, ldw,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_dw_reduce(const float* part, int S, int O, int I, float* dst, int ldw, int accumulate,
                            hipStream_t st) {
  const int64_t n = (int64_t)O * I;
  hipLaunchKernelGGL(dw_reduce_kernel, dim3((unsigned)((n + 63) / 64)), dim3(NT), 0, st, part, S, O, I, dst, ldw,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_vec_reduce(const float* vpart, int nwg, int nvec, const VecSeg* segs, int nseg, float* dparams,
                             int accumulate, hipStream_t st) {
  VecSegs s;
  s.n = nseg;
  for (int i = 0; i < nseg && i < 4; ++i) s.s[i] = segs[i];
  hipLaunchKernelGGL(vec_reduce_kernel, dim3((nvec + 63) / 64), dim3(NT), 0, st, vpart, nwg, nvec, s, dparams,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_mse(const float* out, const float* target, const uint8_t* mask, int64_t n, int d,
                      int64_t global_rows, float* loss, float* d_out, hipStream_t st) {
  // loss[1] doubles as scratch for the gradient scale: scale is written to loss+1.
  // Large inputs: per-workgroup partials first, parked in d_out (overwritten
  // by the gradient afterwards).
  if (n * d >= 4 * MSE_G) {
    uint32_t* scratch = reinterpret_cast<uint32_t*>(d_out);
    hipLaunchKernelGGL(mse_partial_kernel, dim3(MSE_G), dim3(NT), 0, st, out, target, mask, n, d, scratch);
    hipLaunchKernelGGL(mse_final_kernel, dim3(1), dim3(64), 0, st, scratch, d, global_rows, loss, loss + 1);
  } else {
    hipLaunchKernelGGL(mse_loss_kernel, dim3(1), dim3(NT), 0, st, out, target, mask, n, d, global_rows, loss,
                       loss + 1);
  }
  if (n > 0)
    hipLaunchKernelGGL(mse_grad_kernel, dim3((unsigned)((n * d + NT - 1) / NT)), dim3(NT), 0, st, out, target, mask,
                       n, d, loss + 1, d_out);
  return hipGetLastError();
}

}  // namespace mgn
