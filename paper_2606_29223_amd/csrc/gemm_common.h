// Pieces of the skinny-M decode GEMM shared by every kernel that runs it:
// the 16-byte fragment types and their MFMA steps, the weight and
// activation loads, and the split-K reduction with the residual epilogue.
// A kernel that multiplies a weight tile through these gets the same bits
// as the stand-alone decode GEMM for the same tile and rows.
#pragma once

#include "dex_kernels.h"

namespace dex {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4_t;

__device__ __forceinline__ float bf2f(bf16 b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ bf16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16)(u >> 16);
}
template <typename T> __device__ __forceinline__ T to_t(float f);
template <> __device__ __forceinline__ float to_t<float>(float f) { return f; }
template <> __device__ __forceinline__ bf16 to_t<bf16>(float f) { return f2bf(f); }

// One 16-byte fragment per lane and the MFMA steps it feeds.
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  u32x4_t v;
  static constexpr int EPB = 8;           // elements per 16 bytes
  __device__ __forceinline__ static f32x4_t mma(const Frag &a, const Frag &b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                   __builtin_bit_cast(bf16x8_t, b.v), c, 0, 0, 0);
  }
};
template <> struct Frag<float> {
  u32x4_t v;
  static constexpr int EPB = 4;
  __device__ __forceinline__ static f32x4_t mma(const Frag &a, const Frag &b, f32x4_t c) {
    // k-slot (lane group g, element e) <-> k = 4 g + e, identical for A and B
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v.x), __uint_as_float(b.v.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v.y), __uint_as_float(b.v.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v.z), __uint_as_float(b.v.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v.w), __uint_as_float(b.v.w), c, 0, 0, 0);
    return c;
  }
};

__device__ __forceinline__ u32x4_t load16(const void *p, bool ok) {
  if (!ok) return u32x4_t{0u, 0u, 0u, 0u};
  return __builtin_nontemporal_load((const u32x4_t *)p);
}
__device__ __forceinline__ u32x4_t load16_cached(const void *p, bool ok) {
  if (!ok) return u32x4_t{0u, 0u, 0u, 0u};
  return *(const u32x4_t *)p;
}

// RMSNorm reciprocal scale of one row from its sum-of-squares partials.  The
// single definition used by every consumer: lane j sums partials j, j+64, ...
// in order, then a fixed butterfly across the wave.
__device__ __forceinline__ float row_rscale(const float *part, int n_part, float inv_d, float eps, int lane) {
  float s = 0.f;
  for (int t = lane; t < n_part; t += 64) s += part[t];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  return 1.0f / sqrtf(s * inv_d + eps);
}

// The eight waves' split-K partials of one weight block meet in LDS and are
// summed in wave order; vt[nl][ml] is then output column nl (of the tile)
// for row ml of the block.  red: [GEMM_WAVES][64][4] floats of this block.
template <int MB>
__device__ __forceinline__ void reduce_block(const float (*red)[MB][64][4], float (*vt)[16 * MB]) {
  for (int e = threadIdx.x; e < MB * 256; e += GEMM_THREADS) {
    const int mb = e / 256, li = e % 256;
    const int ln = li >> 2, i = li & 3;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < GEMM_WAVES; ++w) sum += red[w][mb][ln][i];
    // C layout: lane ln holds rows 4*(ln/16)+i (output columns) of column ln%16 (input rows)
    const int nl = 4 * (ln >> 4) + i;
    const int ml = mb * 16 + (ln & 15);
    vt[nl][ml] = sum;
  }
}

// RESID epilogue of one 16-column tile for rows m0 .. m0 + Mloc: h += alpha *
// acc (+ bias), the next RMSNorm's input g * h in the matrix-core type, and the
// tile's sum-of-squares partial of each row; with row_bnd the results go to
// the rows' boundary storage instead.  sq: [16][16 * MB] LDS scratch.  Ends
// with a workgroup barrier.
template <typename T, int MB>
__device__ __forceinline__ void epi_resid(const GemmArgs &a, int tile, int m0, int Mloc,
                                          const float (*vt)[16 * MB], float (*sq)[16 * MB]) {
  for (int e = threadIdx.x; e < 16 * Mloc; e += GEMM_THREADS) {
    const int ml = e / 16, nl = e % 16;
    const int m = m0 + ml, n = tile * 16 + nl;
    const float *hin = a.h + (size_t)m * a.ld_h;
    float *hout = (a.row_bnd != nullptr) ? a.bnd_h + (size_t)a.row_bnd[m] * a.ld_h : a.h + (size_t)m * a.ld_h;
    const float br = (a.bias != nullptr) ? a.alpha * (vt[nl][ml] + a.bias[n]) : a.alpha * vt[nl][ml];
    const float hn = hin[n] + br;
    hout[n] = hn;
    if (a.xb != nullptr) ((T *)a.xb)[(size_t)m * a.ld_h + n] = to_t<T>(a.g_next[n] * hn);
    sq[nl][ml] = hn * hn;
  }
  __syncthreads();
  for (int ml = threadIdx.x; ml < Mloc; ml += GEMM_THREADS) {
    const int m = m0 + ml;
    float s = 0.f;
#pragma unroll
    for (int nl = 0; nl < 16; ++nl) s += sq[nl][ml];
    float *po = (a.row_bnd != nullptr) ? a.bnd_part + (size_t)a.row_bnd[m] * a.n_part_out
                                       : a.part_out + (size_t)m * a.n_part_out;
    po[tile] = s;
  }
}

}  // namespace dex
