// Small kernels of the decode round: stage input (embedding gather or
// boundary restore), argmax reduction, verify/commit, key/value collapse
// gather, and a plain copy used to calibrate traffic counters.
#include "dex_kernels.h"

namespace dex {

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
template <typename T>
__global__ __launch_bounds__(256) void prep_kernel(PrepArgs a) {
  const int m = blockIdx.x;
  const int mo = (a.row_out != nullptr) ? a.row_out[m] : m;
  float *h = a.h + (size_t)mo * a.d;
  float *part = a.part + (size_t)mo * a.n_part;
  T *xb = (T *)a.xb + (size_t)mo * a.d;
  if (a.from_embed) {
    const T *e = (const T *)a.embed + (size_t)a.row_tok[m] * a.d;
    for (int i = threadIdx.x; i < a.d; i += blockDim.x) {
      float v;
      if constexpr (sizeof(T) == 2) v = bf2f_m(e[i]);
      else v = e[i];
      h[i] = v;
      if (xb != nullptr) {
        if constexpr (sizeof(T) == 2) xb[i] = f2bf_m(a.g[i] * v);
        else xb[i] = a.g[i] * v;
      }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < a.n_part; t += blockDim.x) {
      float s = 0.f;
      for (int j = 0; j < 16; ++j) {
        const float v = h[16 * t + j];
        s += v * v;
      }
      part[t] = s;
    }
  } else {
    const float *bh = a.bnd_h + (size_t)a.row_src[m] * a.d;
    const float *bp = a.bnd_part + (size_t)a.row_src[m] * a.n_part;
    for (int i = threadIdx.x; i < a.d; i += blockDim.x) {
      const float v = bh[i];
      h[i] = v;
      if (xb != nullptr) {
        if constexpr (sizeof(T) == 2) xb[i] = f2bf_m(a.g[i] * v);
        else xb[i] = a.g[i] * v;
      }
    }
    for (int t = threadIdx.x; t < a.n_part; t += blockDim.x) part[t] = bp[t];
  }
}

hipError_t launch_prep(int dtype, const PrepArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (dtype == 1) hipLaunchKernelGGL(prep_kernel<bf16>, dim3(a.M), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(prep_kernel<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

// argmax over the per-tile winners of each row; the lowest id wins ties.
// Lane j scans a contiguous run of tiles in order, then a butterfly under the
// total order (value, -id): the result is the sequential argmax.
__global__ __launch_bounds__(64) void argmax_kernel(ArgmaxArgs a) {
  const int m = blockIdx.x, lane = threadIdx.x;
  const float2 *src = a.amax + (size_t)m * a.n_tiles;
  const int per = (a.n_tiles + 63) / 64;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int t = lane * per; t < min(a.n_tiles, (lane + 1) * per); ++t) {
    const float v = src[t].x;
    const int i = __float_as_int(src[t].y);
    if (v > bv || (v == bv && i < bi)) { bv = v; bi = i; }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
  }
  if (lane == 0) {
    a.u_out[m] = bi;
    if (a.cand != nullptr) a.cand[a.row_cand[m]] = bi;
  }
}

hipError_t launch_argmax(const ArgmaxArgs &a, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(a.M), dim3(64), 0, s, a);
  return hipGetLastError();
}

// Validate and commit (Section 3.2, commit process): the anchor's candidates
// u_0..u_{N-1} by increasing depth; the committed token is u_{N-1}; the
// reusable branch is the shallowest k <= N-2 with u_k == u_{N-1}, else N-1.
__global__ void commit_kernel(CommitArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int *u = a.cand + a.seq_cand[i];
  const int y = u[a.N - 1];
  int k = a.N - 1;
  for (int j = 0; j < a.N - 1; ++j)
    if (u[j] == y) { k = j; break; }
  a.out[2 * i] = y;
  a.out[2 * i + 1] = k;
}

hipError_t launch_commit(const CommitArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kernel, dim3((a.n + 63) / 64), dim3(64), 0, s, a);
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
