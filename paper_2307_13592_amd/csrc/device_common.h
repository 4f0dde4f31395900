// Device-side building blocks shared by the libmgn kernels (gfx950 / CDNA4).
//
//  - bf16 storage as raw 16-bit words, round-to-nearest-even conversion;
//  - the two MFMA precisions (fp32: v_mfma_f32_16x16x4_f32, bf16:
//    v_mfma_f32_16x16x32_bf16), with weights pre-packed so that one wave's
//    B fragment for one (16-column block, k-group) is 1 KiB of contiguous
//    memory (64 lanes x 16 bytes);
//  - a wave-level tile GEMM reading the A operand from LDS.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mgn {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint16_t f2bf(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 path: 16x16x4 MFMA; a 16-byte fragment per lane holds 4 consecutive
// k values, consumed by 4 MFMAs (k-group of 16).
struct PF32 {
  using T = float;
  static constexpr int KG = 16;   // k values per k-group
  static constexpr int EL = 4;    // elements per lane per 16-byte fragment
  static constexpr int PAD = 4;   // LDS row padding (elements)
  __device__ __forceinline__ static T cvt(float x) { return x; }
  __device__ __forceinline__ static float tof(T x) { return x; }
  __device__ __forceinline__ static void mma(floatx4& c, const uint4& a, const uint4& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  }
};

// bf16 path: 16x16x32 MFMA, 8 bf16 per lane per fragment, fp32 accumulate.
struct PBF16 {
  using T = uint16_t;
  static constexpr int KG = 32;
  static constexpr int EL = 8;
  static constexpr int PAD = 8;
  __device__ __forceinline__ static T cvt(float x) { return f2bf(x); }
  __device__ __forceinline__ static float tof(T x) { return bf2f(x); }
  __device__ __forceinline__ static void mma(floatx4& c, const uint4& a, const uint4& b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
  }
};

// Linear layer as the kernels see it.  wf: packed for Y = X W^T (B[k][j] =
// W[j][k], k over `in`); wb: packed for dX = dY W (B[k][j] = W[k][j], k over
// `out`).  Packed layout: [n-block][k-group][lane][EL], lane = j%16 + 16*q,
// element e holds k = kgroup*KG + q*EL + e.
struct Lin {
  const uint4* wf;
  const uint4* wb;
  const float* b;
  int in, out;
  int nkgf, nkgb;  // k-groups of the forward / backward packing
};

struct Mlp {
  Lin lin[3];
  const float* gamma;  // null: no LayerNorm (decoder)
  const float* beta;
  int depth;
};

// acc[m][n] = sum_k A[m*16 + i][k] * B[k][n*16 + j] over the wave's n-blocks
// nb0 .. nb0+NBW-1, for MB row blocks of A (row-major in LDS, lda elements).
template <class P, int MB, int NBW>
__device__ __forceinline__ void wave_gemm(const typename P::T* A, int lda, const uint4* __restrict__ Bp, int nkg,
                                          int nb0, floatx4 (&acc)[MB][NBW]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int n = 0; n < NBW; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};
  const typename P::T* Ar = A + (lane & 15) * lda + (lane >> 4) * P::EL;
  const uint4* Bl = Bp + (size_t)nb0 * nkg * 64 + lane;
  uint4 bnext[NBW];
#pragma unroll
  for (int n = 0; n < NBW; ++n) bnext[n] = Bl[(size_t)n * nkg * 64];
  for (int kg = 0; kg < nkg; ++kg) {
    uint4 b[NBW];
#pragma unroll
    for (int n = 0; n < NBW; ++n) b[n] = bnext[n];
    if (kg + 1 < nkg) {
#pragma unroll
      for (int n = 0; n < NBW; ++n) bnext[n] = Bl[((size_t)n * nkg + kg + 1) * 64];
    }
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const uint4 a = *reinterpret_cast<const uint4*>(Ar + m * 16 * lda + kg * P::KG);
#pragma unroll
      for (int n = 0; n < NBW; ++n) P::mma(acc[m][n], a, b[n]);
    }
  }
}

// Same with the number of k-groups known at compile time, software
// pipelined: B fragments are fetched PF k-groups ahead (a ring of registers),
// A fragments one k-group ahead, so neither global nor LDS latency is waited
// on inside the loop.  ZERO = false accumulates onto acc.
// STRIDE: k-groups per 16-column block of the packed layer (NKG unless the
// product uses a k-range of a wider layer, Bp then pointing at its start).
template <class P, int MB, int NBW, int NKG, bool ZERO = true, int STRIDE = NKG>
__device__ __forceinline__ void wave_gemm_k(const typename P::T* A, int lda, const uint4* __restrict__ Bp, int nb0,
                                            floatx4 (&acc)[MB][NBW]) {
  constexpr int PFW = NBW >= 4 ? 2 : (NBW == 2 ? 4 : 6);  // at most ~8 fragments in flight
  constexpr int PF = NKG < PFW ? NKG : PFW;
  const int lane = threadIdx.x & 63;
  if constexpr (ZERO) {
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int n = 0; n < NBW; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  const typename P::T* Ar = A + (lane & 15) * lda + (lane >> 4) * P::EL;
  const uint4* Bl = Bp + (size_t)nb0 * STRIDE * 64 + lane;
  uint4 b[PF][NBW];
#pragma unroll
  for (int p = 0; p < PF; ++p)
#pragma unroll
    for (int n = 0; n < NBW; ++n) b[p][n] = Bl[(n * STRIDE + p) * 64];
  uint4 a[2][MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) a[0][m] = *reinterpret_cast<const uint4*>(Ar + m * 16 * lda);
#pragma unroll
  for (int kg = 0; kg < NKG; ++kg) {
    uint4 bc[NBW];
#pragma unroll
    for (int n = 0; n < NBW; ++n) bc[n] = b[kg % PF][n];
    if (kg + PF < NKG) {
#pragma unroll
      for (int n = 0; n < NBW; ++n) b[kg % PF][n] = Bl[(n * STRIDE + kg + PF) * 64];
    }
    if (kg + 1 < NKG) {
#pragma unroll
      for (int m = 0; m < MB; ++m)
        a[(kg + 1) & 1][m] = *reinterpret_cast<const uint4*>(Ar + m * 16 * lda + (kg + 1) * P::KG);
    }
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int n = 0; n < NBW; ++n) P::mma(acc[m][n], a[kg & 1][m], bc[n]);
  }
}

// One 16-column block with the layer's B fragments held in registers (all
// NKG k-groups, loaded once per kernel); A comes from LDS, one k-group ahead.
template <class P, int MB, int NKG>
__device__ __forceinline__ void wave_gemm_w(const typename P::T* A, int lda, const uint4 (&w)[NKG],
                                            floatx4 (&acc)[MB]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m] = floatx4{0.f, 0.f, 0.f, 0.f};
  const typename P::T* Ar = A + (lane & 15) * lda + (lane >> 4) * P::EL;
  uint4 a[2][MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) a[0][m] = *reinterpret_cast<const uint4*>(Ar + m * 16 * lda);
#pragma unroll
  for (int kg = 0; kg < NKG; ++kg) {
    if (kg + 1 < NKG) {
#pragma unroll
      for (int m = 0; m < MB; ++m)
        a[(kg + 1) & 1][m] = *reinterpret_cast<const uint4*>(Ar + m * 16 * lda + (kg + 1) * P::KG);
    }
#pragma unroll
    for (int m = 0; m < MB; ++m) P::mma(acc[m], a[kg & 1][m], w[kg]);
  }
}

// Loads the B fragments of 16-column block nb (all NKG k-groups) of a packed layer.
template <int NKG>
__device__ __forceinline__ void load_block(const uint4* __restrict__ Bp, int nb, uint4 (&w)[NKG]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int kg = 0; kg < NKG; ++kg) w[kg] = Bp[((size_t)nb * NKG + kg) * 64 + lane];
}

// Row / column of accumulator element r (0..3) of a 16x16 MFMA block for
// this lane: row 4*(lane/16) + r, column lane%16.
__device__ __forceinline__ int acc_row(int r) { return ((threadIdx.x & 63) >> 4) * 4 + r; }
__device__ __forceinline__ int acc_col() { return threadIdx.x & 15; }

// Static, XCD-aware assignment of `ntiles` tiles to a persistent grid: the
// grid's blocks are dealt round-robin to the 8 XCDs, so block b works on the
// b%8-th contiguous eighth of the tiles and neighbouring tiles share an L2.
struct TileIter {
  int t, end, stride;
  __device__ TileIter(int ntiles, int first = 0) {
    const int x = blockIdx.x & 7, q = blockIdx.x >> 3, nq = gridDim.x >> 3;
    const int lo = (int)(((int64_t)ntiles * x) >> 3), hi = (int)(((int64_t)ntiles * (x + 1)) >> 3);
    t = first + lo + q;
    end = first + hi;
    stride = nq;
  }
  __device__ bool valid() const { return t < end; }
  __device__ void next() { t += stride; }
};

}  // namespace mgn
