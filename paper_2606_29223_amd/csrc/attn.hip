// Branch-masked attention over a shared-prefix key/value cache (gfx950).
//
// A row (one lattice node, or one prompt position during prefill) at
// absolute position pos attends to the logical keys 0..pos of its own
// prefix: positions [0, nc) are committed cache entries (shared by every row
// of the sequence), positions [nc, pos] are the entries of its ancestor slots
// and its own slot, listed in `chain`.  Grouped-query heads: query head h
// reads key/value head h / (H / Hkv).
//
// Work split: one workgroup per (row group, kv head, split of 256 logical
// keys).  A row group is up to 64 / (H/Hkv) rows of one sequence; the
// committed keys of a 64-key tile are staged in LDS once and shared by all
// rows and all query heads of the group.  Each wave owns (row, head) pairs;
// a lane owns one key of the tile for the scores and head dimensions lane
// and lane + 64 for the value sum.  Online softmax across the split's tiles,
// then a separate combine over splits.
//
// Every quantity a row computes depends only on its logical key sequence:
// split and tile boundaries are fixed logical positions, each dot product
// and each value sum runs in key/dimension order through one code path
// whether the key is read from LDS or from a chain entry, and the combine
// walks splits in order.  So a node evaluated speculatively (tail keys in
// lattice slots) gets the bits plain decoding gets at the same position.
#include "dex_kernels.h"

namespace dex {

__device__ __forceinline__ float ld_elem(const float *p) { return *p; }
__device__ __forceinline__ float ld_elem(const bf16 *p) { return __uint_as_float(((uint32_t)*p) << 16); }
__device__ __forceinline__ float bfl(bf16 b) { return __uint_as_float(((uint32_t)b) << 16); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <typename T>
__global__ __launch_bounds__(ATT_THREADS) void attn_kernel(AttnArgs a) {
  constexpr int PAD = (sizeof(T) == 2) ? 2 : 1;    // odd word stride per LDS row
  __shared__ float qs[ATT_MAX_PAIRS][128];
  __shared__ T ks[ATT_TILE][128 + PAD];
  __shared__ T vs[ATT_TILE][128 + PAD];

  const int gi = blockIdx.x, kvh = blockIdx.y, split = blockIdx.z;
  const int r0 = a.grp_row0[gi], nr = a.grp_nrows[gi], seq = a.grp_seq[gi];
  const int hd = a.head_dim;
  const int G = a.n_heads / a.n_kv_heads;
  const int npairs = nr * G;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

  int maxpos = 0, ncmax = 0;
  for (int r = 0; r < nr; ++r) {
    maxpos = max(maxpos, a.row_pos[r0 + r]);
    ncmax = max(ncmax, a.row_nc[r0 + r]);
  }
  const int kbeg = split * ATT_SPLIT;
  if (kbeg > maxpos) return;
  const int kend = min(kbeg + ATT_SPLIT, maxpos + 1);

  // queries of the group's pairs (pair p: row p / G, head kvh * G + p % G)
  for (int e = threadIdx.x; e < npairs * hd; e += ATT_THREADS) {
    const int p = e / hd, i = e % hd;
    const int r = r0 + p / G, h = kvh * G + p % G;
    qs[p][i] = a.q[(size_t)r * a.ldq + h * hd + i];
  }

  const T *kbase = (const T *)a.kc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * hd;
  const T *vbase = (const T *)a.vc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * hd;

  // per-pair running state (pairs p = wave, wave + 4, ...)
  constexpr int PPW = ATT_MAX_PAIRS / 4;
  float m_run[PPW], l_run[PPW], o0[PPW], o1[PPW];
#pragma unroll
  for (int i = 0; i < PPW; ++i) { m_run[i] = -INFINITY; l_run[i] = 0.f; o0[i] = 0.f; o1[i] = 0.f; }

  for (int t0 = kbeg; t0 < kend; t0 += ATT_TILE) {
    __syncthreads();
    // stage committed keys/values [t0, t0 + 64) that exist for some row
    const int tn = max(0, min(ATT_TILE, ncmax - t0));
    for (int e = threadIdx.x; e < tn * hd; e += ATT_THREADS) {
      const int i = e / hd, c = e % hd;
      ks[i][c] = kbase[(size_t)(t0 + i) * hd + c];
      vs[i][c] = vbase[(size_t)(t0 + i) * hd + c];
    }
    __syncthreads();
#pragma unroll
    for (int pi = 0; pi < PPW; ++pi) {
      const int p = wave + 4 * pi;
      if (p >= npairs) break;
      const int r = r0 + p / G;
      const int pos = a.row_pos[r], nc = a.row_nc[r];
      if (t0 > pos) continue;
      const int coff = a.row_chain_off[r];
      // score of key t0 + lane
      const int t = t0 + lane;
      float s = -INFINITY;
      if (t <= pos) {
        const T *kp = (t < nc) ? &ks[lane][0] : kbase + (size_t)a.chain[coff + (t - nc)] * hd;
        float acc = 0.f;
        for (int i = 0; i < hd; ++i) acc = fmaf(qs[p][i], ld_elem(kp + i), acc);
        s = acc * a.scale;
      }
      const float mt = wave_max(s);
      const float mn = fmaxf(m_run[pi], mt);
      const float c = expf(m_run[pi] - mn);
      const float e = (t <= pos) ? expf(s - mn) : 0.f;
      l_run[pi] = l_run[pi] * c + wave_sum(e);
      float a0 = o0[pi] * c, a1 = o1[pi] * c;
      const int nk = min(ATT_TILE, pos + 1 - t0);
      for (int j = 0; j < nk; ++j) {
        const float ej = __shfl(e, j, 64);
        const int tj = t0 + j;
        const T *vp = (tj < nc) ? &vs[j][0] : vbase + (size_t)a.chain[coff + (tj - nc)] * hd;
        if (lane < hd) a0 = fmaf(ej, ld_elem(vp + lane), a0);
        if (lane + 64 < hd) a1 = fmaf(ej, ld_elem(vp + lane + 64), a1);
      }
      o0[pi] = a0;
      o1[pi] = a1;
      m_run[pi] = mn;
    }
  }
  // partials: o[hd], m, l
#pragma unroll
  for (int pi = 0; pi < PPW; ++pi) {
    const int p = wave + 4 * pi;
    if (p >= npairs) break;
    const int r = r0 + p / G, h = kvh * G + p % G;
    if (a.row_pos[r] < kbeg) continue;
    float *dst = a.part + (((size_t)r * a.n_heads + h) * a.jmax + split) * (hd + 2);
    if (lane < hd) dst[lane] = o0[pi];
    if (lane + 64 < hd) dst[lane + 64] = o1[pi];
    if (lane == 0) { dst[hd] = m_run[pi]; dst[hd + 1] = l_run[pi]; }
  }
}


// out[r][h] = sum_j e^{m_j - M} o_j / sum_j e^{m_j - M} l_j over the splits
// j = 0 .. pos/256 of row r, in split order.
template <typename T>
__global__ __launch_bounds__(128) void combine_kernel(CombineArgs a) {
  const int r = blockIdx.x, h = blockIdx.y, i = threadIdx.x;
  const int hd = a.head_dim;
  const int nsplit = a.row_pos[r] / ATT_SPLIT + 1;
  const float *src = a.part + ((size_t)r * a.n_heads + h) * a.jmax * (hd + 2);
  float M = -INFINITY;
  for (int j = 0; j < nsplit; ++j) M = fmaxf(M, src[j * (hd + 2) + hd]);
  float o = 0.f, l = 0.f;
  for (int j = 0; j < nsplit; ++j) {
    const float w = expf(src[j * (hd + 2) + hd] - M);
    l = fmaf(w, src[j * (hd + 2) + hd + 1], l);
    if (i < hd) o = fmaf(w, src[j * (hd + 2) + i], o);
  }
  if (i < hd) {
    const float v = o / l;
    T *out = (T *)a.out + (size_t)r * a.ld_out + h * hd + i;
    if constexpr (sizeof(T) == 2) {
      uint32_t u = __float_as_uint(v);
      u += 0x7fffu + ((u >> 16) & 1u);
      *out = (T)(u >> 16);
    } else {
      *out = v;
    }
  }
}

hipError_t launch_attention(int dtype, const AttnArgs &a, int n_groups, hipStream_t s) {
  if (a.head_dim > 128 || n_groups <= 0) return hipErrorInvalidValue;
  dim3 grid(n_groups, a.n_kv_heads, a.jmax);
  if (dtype == 1) hipLaunchKernelGGL(attn_kernel<bf16>, grid, dim3(ATT_THREADS), 0, s, a);
  else hipLaunchKernelGGL(attn_kernel<float>, grid, dim3(ATT_THREADS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_combine(int dtype, const CombineArgs &a, int rows, hipStream_t s) {
  if (rows <= 0) return hipErrorInvalidValue;
  dim3 grid(rows, a.n_heads);
  if (dtype == 1) hipLaunchKernelGGL(combine_kernel<bf16>, grid, dim3(128), 0, s, a);
  else hipLaunchKernelGGL(combine_kernel<float>, grid, dim3(128), 0, s, a);
  return hipGetLastError();
}

}  // namespace dex
