// Small kernels of the decode round: stage input (embedding gather or
// boundary restore), argmax reduction with the verify/commit of completed
// anchors, key/value collapse gather, and a plain copy used to calibrate
// traffic counters.
#include "dex_kernels.h"

namespace dex {

constexpr int PREP_THREADS = 64;              // 16-column groups per prep workgroup

__device__ __forceinline__ float bf2f_m(bf16 b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ bf16 f2bf_m(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16)(u >> 16);
}

// Stage input for each row: h (float), its per-16-column sum-of-squares
// partials, and the first RMSNorm's input g*h in the matrix-core type.  Rows
// entering at stage 0 read the embedding (partials computed here); rows
// continuing a slot restore the boundary state saved when the slot finished
// its previous stage (partials copied unchanged, so a layer's norm sees the
// same bits whether or not a stage boundary lies before it).
//
// Thread t of a row owns the 16-column group t: every load of the group is
// requested before anything is stored, so a row costs one memory round trip.
template <typename T>
__global__ __launch_bounds__(PREP_THREADS) void prep_kernel(PrepArgs a) {
  constexpr int EPV = 16 / (int)sizeof(T);     // elements per 16-byte vector
  const int m = blockIdx.x;
  const bool from_embed = m < a.embed_rows;
  const float *gain = a.g;
  if (a.n_seg > 0) {
    int k = 0;
#pragma unroll
    for (int i = 0; i < MAX_SEGS - 1; ++i) k += (i < a.n_seg - 1 && m >= a.seg_end[i]) ? 1 : 0;
    gain = a.seg_g[k];
  }
  const int t = blockIdx.y * PREP_THREADS + threadIdx.x;
  if (t >= a.n_part) return;
  const int mo = (a.row_out != nullptr) ? a.row_out[m] : m;
  const int c0 = 16 * t;
  float v[16], g[16];
  float pin = 0.f;
  if (from_embed) {
    const uint4 *e = (const uint4 *)((const T *)a.embed + (size_t)a.row_tok[m] * a.d + c0);
    uint4 raw[16 / EPV];
#pragma unroll
    for (int q = 0; q < 16 / EPV; ++q) raw[q] = e[q];
#pragma unroll
    for (int q = 0; q < 16 / EPV; ++q) {
      const uint32_t w[4] = {raw[q].x, raw[q].y, raw[q].z, raw[q].w};
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        if constexpr (sizeof(T) == 2) v[q * EPV + k] = bf2f_m((bf16)((w[k >> 1] >> (16 * (k & 1))) & 0xffffu));
        else v[q * EPV + k] = __uint_as_float(w[k]);
      }
    }
  } else {
    const float4 *bh = (const float4 *)(a.bnd_h + (size_t)a.row_src[m] * a.d + c0);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 x = bh[q];
      v[4 * q] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
    }
    pin = a.bnd_part[(size_t)a.row_src[m] * a.n_part + t];
  }
  const float4 *gp = (const float4 *)(gain + c0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 x = gp[q];
    g[4 * q] = x.x; g[4 * q + 1] = x.y; g[4 * q + 2] = x.z; g[4 * q + 3] = x.w;
  }
  float4 *h = (float4 *)(a.h + (size_t)mo * a.d + c0);
#pragma unroll
  for (int q = 0; q < 4; ++q) h[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  if (a.xb != nullptr) {
    uint4 *xb = (uint4 *)((T *)a.xb + (size_t)mo * a.d + c0);
#pragma unroll
    for (int q = 0; q < 16 / EPV; ++q) {
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (sizeof(T) == 2) {
          const int e0 = q * EPV + 2 * k;
          w[k] = (uint32_t)f2bf_m(g[e0] * v[e0]) | ((uint32_t)f2bf_m(g[e0 + 1] * v[e0 + 1]) << 16);
        } else {
          w[k] = __float_as_uint(g[q * EPV + k] * v[q * EPV + k]);
        }
      }
      xb[q] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
  if (from_embed) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) s += v[j] * v[j];
    pin = s;
  }
  a.part[(size_t)mo * a.n_part + t] = pin;
}

hipError_t launch_prep(int dtype, const PrepArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.d % 16 != 0 || a.n_part * 16 != a.d) return hipErrorInvalidValue;
  if (a.n_seg < 0 || a.n_seg > MAX_SEGS || (a.n_seg > 0 && a.seg_end[a.n_seg - 1] != a.M)) return hipErrorInvalidValue;
  const dim3 grid(a.M, (a.n_part + PREP_THREADS - 1) / PREP_THREADS);
  if (dtype == 1) hipLaunchKernelGGL(prep_kernel<bf16>, grid, dim3(PREP_THREADS), 0, s, a);
  else hipLaunchKernelGGL(prep_kernel<float>, grid, dim3(PREP_THREADS), 0, s, a);
  return hipGetLastError();
}

// argmax over the per-tile winners of each row; the lowest id wins ties.
// The order (value, -id) is total, so any reduction order gives the
// sequential argmax: thread j takes tiles j, j + 256, ... (all requested
// before any is compared), then a wave butterfly and a pass over the waves.
__device__ __forceinline__ void amax_take(float &bv, int &bi, float v, int i) {
  if (v > bv || (v == bv && i < bi)) { bv = v; bi = i; }
}
constexpr int AMAX_THREADS = 256;
constexpr int AMAX_PER = 8;                    // tiles per thread per pass
__global__ __launch_bounds__(AMAX_THREADS) void argmax_kernel(ArgmaxArgs a) {
  __shared__ float sv[AMAX_THREADS / 64];
  __shared__ int si[AMAX_THREADS / 64];
  const int m = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float2 *src = a.amax + (size_t)m * a.n_tiles;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int t0 = 0; t0 < a.n_tiles; t0 += AMAX_THREADS * AMAX_PER) {
    float2 x[AMAX_PER];
#pragma unroll
    for (int k = 0; k < AMAX_PER; ++k) {
      const int t = t0 + k * AMAX_THREADS + tid;
      x[k] = t < a.n_tiles ? src[t] : make_float2(-INFINITY, __int_as_float(0x7fffffff));
    }
#pragma unroll
    for (int k = 0; k < AMAX_PER; ++k) amax_take(bv, bi, x[k].x, __float_as_int(x[k].y));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax_take(bv, bi, __shfl_xor(bv, o, 64), __shfl_xor(bi, o, 64));
  if (lane == 0) { sv[wave] = bv; si[wave] = bi; }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < AMAX_THREADS / 64; ++w) amax_take(bv, bi, sv[w], si[w]);
    a.u_out[m] = bi;
    if (a.cand != nullptr) a.cand[a.row_cand[m]] = bi;
    // Validate and commit (Section 3.2, commit process) when this row is an
    // anchor's final-depth node: its candidates u_0..u_{N-2} (earlier rounds)
    // and u_{N-1} = bi; the committed token is u_{N-1}, the reusable branch
    // the shallowest k <= N-2 with u_k == u_{N-1}, else N-1.
    if (a.row_commit != nullptr && a.row_commit[m] >= 0) {
      const int *u = a.cand + a.row_cand[m] - (a.N - 1);
      int k = a.N - 1;
      for (int j = 0; j < a.N - 1; ++j)
        if (u[j] == bi) { k = j; break; }
      a.commit_out[2 * a.row_commit[m]] = bi;
      a.commit_out[2 * a.row_commit[m] + 1] = k;
    }
  }
}

hipError_t launch_argmax(const ArgmaxArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(a.M), dim3(AMAX_THREADS), 0, s, a);
  return hipGetLastError();
}

// Collapse gather.  Job (seq, src entry, dst entry, src slot, dst slot, kind):
// copy the keys/values of one cache entry (every layer, every kv head) and,
// for kind 1, the slot's boundary state and candidate list.  The old anchor
// goes to its committed position (kind 0); retained slots move to the
// other half of the lattice region in canonical order (kind 1), so source
// and destination never overlap.
template <int ELEM>
__global__ __launch_bounds__(256) void collapse_kernel(CollapseArgs a) {
  const int jb = blockIdx.x, l = blockIdx.y;
  const int *j = a.job + 6 * jb;
  const int seq = j[0], se = j[1], de = j[2], ss = j[3], ds = j[4], kind = j[5];
  if (l < a.n_layers) {
    const int n16 = a.head_dim * ELEM / 16;
    for (int e = threadIdx.x; e < a.n_kv_heads * n16; e += blockDim.x) {
      const int g = e / n16, c = e % n16;
      const size_t row = (((size_t)l * a.batch + seq) * a.n_kv_heads + g) * a.kv_entries;
      const size_t bytes_row = (size_t)a.head_dim * ELEM;
      uint4 *kd = (uint4 *)((char *)a.kc + (row + de) * bytes_row) + c;
      const uint4 *ksrc = (const uint4 *)((const char *)a.kc + (row + se) * bytes_row) + c;
      uint4 *vd = (uint4 *)((char *)a.vc + (row + de) * bytes_row) + c;
      const uint4 *vsrc = (const uint4 *)((const char *)a.vc + (row + se) * bytes_row) + c;
      *kd = *ksrc;
      *vd = *vsrc;
    }
  } else if (kind == 1) {
    const size_t sb = (size_t)seq * a.slots2 + ss, db = (size_t)seq * a.slots2 + ds;
    for (int i = threadIdx.x; i < a.d; i += blockDim.x) a.bnd_h[db * a.d + i] = a.bnd_h[sb * a.d + i];
    for (int i = threadIdx.x; i < a.n_part; i += blockDim.x)
      a.bnd_part[db * a.n_part + i] = a.bnd_part[sb * a.n_part + i];
    for (int i = threadIdx.x; i < a.N; i += blockDim.x) a.cand[db * a.N + i] = a.cand[sb * a.N + i];
  }
}

hipError_t launch_collapse(const CollapseArgs &a, hipStream_t s) {
  if (a.n_jobs <= 0) return hipSuccess;
  dim3 grid(a.n_jobs, a.n_layers + 1);
  if (a.elem_bytes == 2) hipLaunchKernelGGL(collapse_kernel<2>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(collapse_kernel<4>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void copy_kernel(uint4 *dst, const uint4 *src, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

__global__ __launch_bounds__(256) void gumbel_kernel(unsigned long long seed, int seq, int pos, int V, float *out) {
  const int v = blockIdx.x * 256 + threadIdx.x;
  if (v < V) out[v] = gumbel_noise(gumbel_key(seed, seq, pos), v);
}

hipError_t launch_gumbel(unsigned long long seed, int seq, int pos, int V, float *out, hipStream_t s) {
  if (V <= 0) return hipSuccess;
  hipLaunchKernelGGL(gumbel_kernel, dim3((V + 255) / 256), dim3(256), 0, s, seed, seq, pos, V, out);
  return hipGetLastError();
}

hipError_t launch_copy(void *dst, const void *src, int64_t bytes, hipStream_t s) {
  const int64_t n = bytes / 16;
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint4 *)dst, (const uint4 *)src, n);
  return hipGetLastError();
}

}  // namespace dex
