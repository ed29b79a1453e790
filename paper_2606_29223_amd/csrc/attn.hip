// Branch-masked attention over a shared-prefix key/value cache (gfx950).
//
// A row (one lattice node, or one prompt position during prefill) at
// absolute position pos attends to the logical keys 0..pos of its own
// prefix: positions [0, nc) are committed cache entries (shared by every row
// of the sequence), positions [nc, pos] are the entries of its ancestor slots
// and its own slot, listed in `chain`.  Grouped-query heads: query head h
// reads key/value head h / (H / Hkv).
//
// Decode: the keys are cut into splits of 64 logical positions; a split
// kernel writes one (o, max, sum) partial per (row, query head, split) and
// combine_kernel merges a row's splits.  attn_mfma_kernel (bf16, head_dim 64
// and 128) runs the two products on the matrix cores; attn_kernel (fp32
// models, bf16 head_dim 32) is its VALU form: one workgroup per (row group,
// kv head, split) stages the split's committed keys and values in LDS,
// patches in each row's chain entries, and scores, normalises and sums per
// row with one lane per key and then per value dimension.
//
// Every quantity a row computes depends only on its logical key sequence:
// split and tile boundaries are fixed logical positions, each dot product
// and each value sum runs in a fixed key/dimension order whether the key is
// read from the committed cache or a chain entry, and the combine's order
// depends only on the row's split count.  So a node evaluated speculatively
// (tail keys in lattice slots) gets the bits plain decoding gets at the same
// position.  Splits of 64 keys keep a long context spread over many waves:
// 8192 keys x 8 kv heads x 8 sequences is 9216 waves per layer.
//
// Prefill: prefill_attn128_kernel (head_dim 128) and prefill_attn_kernel
// (head_dim 64) compute causal attention over the prompt's own keys.
#include "attn_decode.h"

namespace dex {


// Element e of a packed row held as 32-bit words (bf16 pairs or floats).
template <typename T> __device__ __forceinline__ float unpack(const uint32_t *w, int e);
template <> __device__ __forceinline__ float unpack<bf16>(const uint32_t *w, int e) {
  const uint32_t u = w[e >> 1];
  return __uint_as_float((e & 1) ? (u & 0xffff0000u) : (u << 16));
}
template <> __device__ __forceinline__ float unpack<float>(const uint32_t *w, int e) { return __uint_as_float(w[e]); }

// A split record element: the split's output in the cache's element type
// (bf16 rounded to nearest even).
template <typename T> __device__ __forceinline__ T rec_elem(float v);
template <> __device__ __forceinline__ float rec_elem<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 rec_elem<bf16>(float v) { return pf_f2bf(v); }
template <typename T> __device__ __forceinline__ float rec_val(T v);
template <> __device__ __forceinline__ float rec_val<float>(float v) { return v; }
template <> __device__ __forceinline__ float rec_val<bf16>(bf16 v) { return __uint_as_float((uint32_t)v << 16); }

// DPL consecutive record elements (one load) as floats; zeros if !ok.
template <typename T, int DPL>
__device__ __forceinline__ void rec_load(const T *p, bool ok, float (&v)[DPL]) {
  if constexpr (DPL == 2 && sizeof(T) == 2) {
    const uint32_t u = ok ? *(const uint32_t *)p : 0u;
    v[0] = __uint_as_float(u << 16);
    v[1] = __uint_as_float(u & 0xffff0000u);
  } else if constexpr (DPL == 2) {
    const float2 f = ok ? *(const float2 *)p : make_float2(0.f, 0.f);
    v[0] = f.x;
    v[1] = f.y;
  } else {
#pragma unroll
    for (int q = 0; q < DPL; ++q) v[q] = ok ? rec_val<T>(p[q]) : 0.f;
  }
}

// One wave per (row group, kv head, split of 64 logical keys).  Lane i owns
// key s0 + i for the scores and head dimensions [i*DPL, i*DPL + DPL) for the
// value sum.
template <typename T, int HD>
__global__ __launch_bounds__(ATT_THREADS) void attn_kernel(AttnArgs a) {
  constexpr int WORDS = HD * (int)sizeof(T) / 4;     // 32-bit words per key row
  constexpr int V4 = WORDS / 4;                      // 16-byte loads per key row
  constexpr int DPL = HD >= 64 ? HD / 64 : 1;        // value dims per lane
  constexpr int GMAX = 8;
  constexpr int KSTRIDE = WORDS + 4;
  constexpr int EPC = 16 / (int)sizeof(T);           // elements per 16-byte chunk
  __shared__ __attribute__((aligned(16))) float qs[GMAX][HD];
  __shared__ __attribute__((aligned(16))) uint32_t ks[ATT_SPLIT][KSTRIDE];
  __shared__ __attribute__((aligned(16))) uint32_t vs[ATT_SPLIT][WORDS];
  __shared__ __attribute__((aligned(16))) float es[GMAX][ATT_SPLIT];

  const int gi = blockIdx.x, kvh = blockIdx.y, split = blockIdx.z;
  const int r0 = a.grp_row0[gi], nr = a.grp_nrows[gi], seq = a.grp_seq[gi];
  const int G = a.n_heads / a.n_kv_heads;
  const int lane = threadIdx.x;
  int maxpos = 0, ncmax = 0;
  for (int r = 0; r < nr; ++r) {
    maxpos = max(maxpos, a.row_pos[r0 + r]);
    ncmax = max(ncmax, a.row_nc[r0 + r]);
  }
  const int s0 = split * ATT_SPLIT;
  if (s0 > maxpos) return;
  const T *kbase = (const T *)a.kc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;
  const T *vbase = (const T *)a.vc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;

  // committed keys and values of the split, loaded together with the first
  // row's queries: each instruction covers four whole key rows (1 KB
  // contiguous), then K goes to one padded LDS row per key (lane i's key
  // row i) and V to the value tile.  Positions past the committed prefix
  // stay zero until a row's chain entries are patched in.
  const int t = s0 + lane;
  uint4 *krow = (uint4 *)&ks[lane][0];
  const int tn = max(0, min(ATT_SPLIT, ncmax - s0));
  // `held` names the key in this lane's LDS row: -2 the committed one at
  // position t, -1 none, else a cache entry of a row's chain
  int held = t - s0 < tn ? -2 : -1;
  constexpr int Q4 = GMAX * HD / 4 / ATT_THREADS;
  float4 qv[Q4];
  auto load_q = [&](int r) {
    const float4 *qsrc = (const float4 *)(a.q + (size_t)r * a.ldq + kvh * G * HD);
#pragma unroll
    for (int i = 0; i < Q4; ++i) {
      const int e = lane + i * ATT_THREADS;
      qv[i] = (e < G * HD / 4) ? qsrc[e] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  {
    constexpr int PER = ATT_SPLIT * V4 / ATT_THREADS;   // 16-byte loads per lane
    uint4 v[PER], k[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane + i * ATT_THREADS, j = e / V4, c = e % V4;
      const bool ok = j < tn;
      k[i] = ok ? ((const uint4 *)(kbase + (size_t)(s0 + j) * HD))[c] : make_uint4(0, 0, 0, 0);
      v[i] = ok ? ((const uint4 *)(vbase + (size_t)(s0 + j) * HD))[c] : make_uint4(0, 0, 0, 0);
    }
    load_q(r0);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = lane + i * ATT_THREADS;
      *((uint4 *)&ks[e / V4][0] + e % V4) = k[i];
      *((uint4 *)&vs[e / V4][0] + e % V4) = v[i];
    }
  }

  for (int rr = 0; rr < nr; ++rr) {
    const int r = r0 + rr;
    const int pos = a.row_pos[r], nc = a.row_nc[r], coff = a.row_chain_off[r];
    if (s0 > pos) continue;
    if (rr > 0) load_q(r);
    __syncthreads();
    {
      float4 *qdst = (float4 *)&qs[0][0];
#pragma unroll
      for (int i = 0; i < Q4; ++i) qdst[lane + i * ATT_THREADS] = qv[i];
    }
    // this row's chain values at positions [max(nc, s0), pos] of the split
    const int tb = max(nc, s0), te = min(pos, s0 + ATT_SPLIT - 1);
    for (int e = lane; e < (te - tb + 1) * V4; e += ATT_THREADS) {
      const int tj = tb + e / V4, c = e % V4;
      *((uint4 *)&vs[tj - s0][0] + c) = ((const uint4 *)(vbase + (size_t)a.chain[coff + (tj - nc)] * HD))[c];
    }
    // this row's key at logical position t: committed, or its own chain
    const bool valid = t <= pos;
    const int want = (t < nc) ? -2 : (valid ? a.chain[coff + (t - nc)] : -1);
    if (want != -1 && want != held) {
      const uint4 *src = (const uint4 *)(kbase + (size_t)(want == -2 ? t : want) * HD);
#pragma unroll
      for (int i = 0; i < V4; ++i) krow[i] = src[i];
      held = want;
    }
    __syncthreads();
    // scores, one independent chain per head, dimensions in order
    float sacc[GMAX];
#pragma unroll
    for (int g = 0; g < GMAX; ++g) sacc[g] = 0.f;
#pragma unroll 2
    for (int c = 0; c < V4; ++c) {
      const uint4 kw = valid ? krow[c] : make_uint4(0, 0, 0, 0);
      const uint32_t w4[4] = {kw.x, kw.y, kw.z, kw.w};
      float kv[EPC];
#pragma unroll
      for (int e2 = 0; e2 < EPC; ++e2) kv[e2] = unpack<T>(w4, e2);
#pragma unroll
      for (int g = 0; g < GMAX; ++g) {
        if (g < G) {
          const float4 *q4 = (const float4 *)&qs[g][c * EPC];
#pragma unroll
          for (int e4 = 0; e4 < EPC / 4; ++e4) {
            const float4 qq = q4[e4];
            sacc[g] = fmaf(qq.x, kv[4 * e4 + 0], sacc[g]);
            sacc[g] = fmaf(qq.y, kv[4 * e4 + 1], sacc[g]);
            sacc[g] = fmaf(qq.z, kv[4 * e4 + 2], sacc[g]);
            sacc[g] = fmaf(qq.w, kv[4 * e4 + 3], sacc[g]);
          }
        }
      }
    }
    float m[GMAX], l[GMAX];
#pragma unroll
    for (int g = 0; g < GMAX; ++g) {
      if (g >= G) break;
      const float sc = valid ? sacc[g] * a.scale : -INFINITY;
      m[g] = wave_max(sc);
      const float e = valid ? expf(sc - m[g]) : 0.f;
      l[g] = wave_sum(e);
      es[g][lane] = e;
    }
    __syncthreads();
    // value sum over the split's 64 keys in position order (weights of keys
    // past pos are exactly zero and their values finite)
    float o[GMAX][DPL];
#pragma unroll
    for (int g = 0; g < GMAX; ++g)
#pragma unroll
      for (int q = 0; q < DPL; ++q) o[g][q] = 0.f;
    const int d0 = lane * DPL;
    const bool dims_ok = d0 < HD;
    const int dsafe = dims_ok ? d0 : 0;
#pragma unroll 4
    for (int j0 = 0; j0 < ATT_SPLIT; j0 += 4) {
      float v[4][DPL];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int q = 0; q < DPL; ++q) v[jj][q] = unpack<T>(&vs[j0 + jj][0], dsafe + q);
#pragma unroll
      for (int g = 0; g < GMAX; ++g) {
        if (g >= G) break;
        const float4 e4 = *(const float4 *)&es[g][j0];
        const float ev[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
#pragma unroll
          for (int q = 0; q < DPL; ++q) o[g][q] = fmaf(ev[jj], v[jj][q], o[g][q]);
      }
    }
#pragma unroll
    for (int g = 0; g < GMAX; ++g) {
      if (g >= G) break;
      const size_t rec = ((size_t)r * a.n_heads + kvh * G + g) * a.jmax + split;
      T *dst = (T *)a.part + rec * HD;
      if (dims_ok) {
#pragma unroll
        for (int q = 0; q < DPL; ++q) dst[d0 + q] = rec_elem<T>(o[g][q]);
      }
      if (lane == 0) { a.stat[2 * rec] = m[g]; a.stat[2 * rec + 1] = l[g]; }
    }
  }

}

// out[r][h] = sum_j w_j o_j / sum_j w_j l_j with w_j = e^{m_j - M},
// M = max_j m_j, over the splits j = 0 .. pos/64 of row r (each split record
// holds its output o_j, in the cache's element type, and its float
// (m_j, l_j)).  One workgroup of CMB_WAVES
// waves per (row, head): wave s sums the splits j = s, s + CMB_WAVES, ... in
// order (lanes over head dimensions) and the wave sums are added in wave
// order; the statistics take one fixed reduction.  The arithmetic depends
// only on the row's split count, never on the other rows of the launch.
// DW head dimensions per workgroup (blockIdx.z picks the slice): each
// dimension's sum is computed the same way whatever the slicing, so a
// launch with few rows splits a head over two workgroups for more latency
// hiding, and the bits do not change.
#ifndef CMB_WAVES
#define CMB_WAVES 4
#endif
template <typename T, int HD, int DW>
__global__ __launch_bounds__(64 * CMB_WAVES) void combine_kernel(CombineArgs a) {
  // dimensions per lane: 4-byte record loads for bf16 (whole heads: 64
  // lanes x 2; half heads: 32 lanes x 2)
  constexpr int DPL = sizeof(T) == 2 ? (DW >= 128 ? DW / 64 : 2) : (DW >= 64 ? DW / 64 : 1);
  constexpr int CH = 16;                       // splits per value chunk
  constexpr int NT = 64 * CMB_WAVES;
  extern __shared__ float ws[];                // [jmax] split weights
  __shared__ float red[CMB_WAVES][DW];         // per-wave weighted sums
  __shared__ float sred[2][CMB_WAVES];         // per-wave max and denominator
  const int r = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, s = tid >> 6;
  const int nsplit = a.row_pos[r] / ATT_SPLIT + 1;
  const int nmine = nsplit > s ? (nsplit - s + CMB_WAVES - 1) / CMB_WAVES : 0;
  const T *src = (const T *)a.part + ((size_t)r * a.n_heads + h) * a.jmax * HD;
  const float *sst = a.stat + ((size_t)r * a.n_heads + h) * a.jmax * 2;
  const int dl = lane * DPL;                   // this lane's first dimension in the slice
  const int d0 = blockIdx.z * DW + dl;
  const bool dok = dl < DW;
  // the split values do not depend on the statistics: the first chunk is
  // requested before them, each next chunk before the current one is summed
  float va[CH][DPL], vb[CH][DPL];
  auto load_chunk = [&](int i0, float (&v)[CH][DPL]) {
#pragma unroll
    for (int jj = 0; jj < CH; ++jj) {
      const int j = s + (i0 + jj) * CMB_WAVES;
      rec_load<T, DPL>(src + (size_t)j * HD + d0, dok && i0 + jj < nmine, v[jj]);
    }
  };
  load_chunk(0, va);
  float M = -INFINITY;
  for (int j = tid; j < nsplit; j += NT) M = fmaxf(M, sst[2 * j]);
  M = wave_max(M);
  if (lane == 0) sred[0][s] = M;
  __syncthreads();
  M = sred[0][0];
#pragma unroll
  for (int w = 1; w < CMB_WAVES; ++w) M = fmaxf(M, sred[0][w]);
  float lp = 0.f;
  for (int j = tid; j < nsplit; j += NT) {
    const float w = expf(sst[2 * j] - M);
    ws[j] = w;
    lp = fmaf(w, sst[2 * j + 1], lp);
  }
  lp = wave_sum(lp);
  if (lane == 0) sred[1][s] = lp;
  __syncthreads();
  float lsum = sred[1][0];
#pragma unroll
  for (int w = 1; w < CMB_WAVES; ++w) lsum += sred[1][w];
  float o[DPL];
#pragma unroll
  for (int q = 0; q < DPL; ++q) o[q] = 0.f;
  auto sum_chunk = [&](int i0, const float (&v)[CH][DPL]) {
#pragma unroll
    for (int jj = 0; jj < CH; ++jj) {
      if (i0 + jj >= nmine) break;
      const float w = ws[s + (i0 + jj) * CMB_WAVES];
#pragma unroll
      for (int q = 0; q < DPL; ++q) o[q] = fmaf(w, v[jj][q], o[q]);
    }
  };
  for (int i0 = 0; i0 < nmine; i0 += 2 * CH) {
    if (i0 + CH < nmine) load_chunk(i0 + CH, vb);
    sum_chunk(i0, va);
    if (i0 + CH >= nmine) break;
    if (i0 + 2 * CH < nmine) load_chunk(i0 + 2 * CH, va);
    sum_chunk(i0 + CH, vb);
  }
  if (dok) {
#pragma unroll
    for (int q = 0; q < DPL; ++q) red[s][dl + q] = o[q];
  }
  __syncthreads();
  if (s != 0 || !dok) return;
  T *out = (T *)a.out + (size_t)r * a.ld_out + h * HD + d0;
#pragma unroll
  for (int q = 0; q < DPL; ++q) {
    float v = red[0][dl + q];
#pragma unroll
    for (int w = 1; w < CMB_WAVES; ++w) v += red[w][dl + q];
    v = v / lsum;
    if constexpr (sizeof(T) == 2) {
      uint32_t u = __float_as_uint(v);
      u += 0x7fffu + ((u >> 16) & 1u);
      out[q] = (T)(u >> 16);
    } else {
      out[q] = v;
    }
  }
}

template <typename T>
static hipError_t launch_attn_t(const AttnArgs &a, dim3 grid, hipStream_t s) {
  switch (a.head_dim) {
    case 32: hipLaunchKernelGGL((attn_kernel<T, 32>), grid, dim3(ATT_THREADS), 0, s, a); break;
    case 64: hipLaunchKernelGGL((attn_kernel<T, 64>), grid, dim3(ATT_THREADS), 0, s, a); break;
    case 128: hipLaunchKernelGGL((attn_kernel<T, 128>), grid, dim3(ATT_THREADS), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t launch_comb_t(const CombineArgs &a, int rows, hipStream_t s) {
  const size_t smem = (size_t)a.jmax * 4;
  const dim3 block(64 * CMB_WAVES);
  switch (a.head_dim) {
    case 32: hipLaunchKernelGGL((combine_kernel<T, 32, 32>), dim3(rows, a.n_heads), block, smem, s, a); break;
    case 64: hipLaunchKernelGGL((combine_kernel<T, 64, 64>), dim3(rows, a.n_heads), block, smem, s, a); break;
    case 128:
      // up to 512 (row, head) pairs: half a head per workgroup (latency-bound
      // launches); beyond, a whole head (bandwidth-bound, fewer statistics reads)
      if ((size_t)rows * a.n_heads <= 512)
        hipLaunchKernelGGL((combine_kernel<T, 128, 64>), dim3(rows, a.n_heads, 2), block, smem, s, a);
      else
        hipLaunchKernelGGL((combine_kernel<T, 128, 128>), dim3(rows, a.n_heads, 1), block, smem, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_combine(int dtype, const CombineArgs &a, int rows, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (a.jmax > ATT_MAX_SPLITS) return hipErrorInvalidValue;
  return dtype == 1 ? launch_comb_t<bf16>(a, rows, s) : launch_comb_t<float>(a, rows, s);
}



// ------------------------------------------------------------------------
// Causal prompt attention on the matrix cores (bf16 keys/values).
//
// Workgroup = (32 query rows, kv head, sequence); wave w is query head
// kvh * G + w.  Key blocks of 64 positions are staged in LDS -- K as
// [key][dim] and V transposed as [dim][key], rows padded so the 16-byte
// operand reads of a wave hit distinct banks -- and each wave runs
//   S = Q K^T   (v_mfma_f32_16x16x32_bf16, 2 x 4 tiles of 16 x 16),
// an online softmax per query row (causal mask on the diagonal block),
//   O += P V    (P rounded to bf16 through a per-wave LDS tile),
// and finally writes O / l.  Only prompt prefill uses it: its results feed
// plain and lattice decoding alike.
// Max and sum over the 16 lanes of a row with DPP moves; the partner order
// (lane ^ 1, lane ^ 2, then the other quad, then the other half-row) adds
// exactly the operands of the xor butterfly, so every lane holds the same bits.
template <int CTRL>
__device__ __forceinline__ float pf_dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, pf_dpp<0xB1>(v));
  v = fmaxf(v, pf_dpp<0x4E>(v));
  v = fmaxf(v, pf_dpp<0x141>(v));
  return fmaxf(v, pf_dpp<0x140>(v));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += pf_dpp<0xB1>(v);
  v += pf_dpp<0x4E>(v);
  v += pf_dpp<0x141>(v);
  return v + pf_dpp<0x140>(v);
}

template <int HD>
__global__ __launch_bounds__(512) void prefill_attn_kernel(PrefillAttnArgs a) {
  constexpr int QB = 32, KB = 64;
  constexpr int KS = HD / 32;          // MFMA k-steps over head dims
  constexpr int DT = HD / 16;          // 16-wide output tiles over head dims
  constexpr int KROW = HD + 8;         // bf16 elements per padded K row
  constexpr int VROW = KB + 8;         // bf16 elements per padded V^T / P row
  __shared__ __attribute__((aligned(16))) uint16_t ks[KB][KROW];
  __shared__ __attribute__((aligned(16))) uint16_t vt[HD][VROW];
  __shared__ __attribute__((aligned(16))) uint16_t pt[8][QB][VROW];

  const int qb = blockIdx.x, kvh = blockIdx.y, seq = blockIdx.z;
  const int G = a.n_heads / a.n_kv_heads;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nthr = blockDim.x;
  const int r16 = lane & 15, grp = lane >> 4;
  const int h = kvh * G + wave;
  const int P = a.prompt_len;
  const int q0 = qb * QB;
  const size_t row_base = (size_t)seq * P;
  const uint16_t *kbase = (const uint16_t *)a.kc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;
  const uint16_t *vbase = (const uint16_t *)a.vc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;

  // Q fragments (A operand): lane holds row r16 of each 16-row tile, dims
  // ks*32 + grp*8 .. +8, rounded to bf16
  pf_bf16x8 qf[2][KS];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    const int row = q0 + mt * 16 + r16;
    const bool ok = row < P;
    const float *src = a.q + (row_base + (ok ? row : 0)) * a.ldq + h * HD;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      uint16_t t[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = ok ? pf_f2bf(src[s * 32 + grp * 8 + e]) : (uint16_t)0;
      uint4 u;
      u.x = t[0] | ((uint32_t)t[1] << 16); u.y = t[2] | ((uint32_t)t[3] << 16);
      u.z = t[4] | ((uint32_t)t[5] << 16); u.w = t[6] | ((uint32_t)t[7] << 16);
      qf[mt][s] = __builtin_bit_cast(pf_bf16x8, u);
    }
  }
  pf_f32x4 o[2][DT];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[mt][dt] = pf_f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun[2][4], lrun[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) { mrun[mt][i] = -INFINITY; lrun[mt][i] = 0.f; }

  const int last_row = min(q0 + QB, P) - 1;
  for (int k0 = 0; k0 <= last_row; k0 += KB) {
    __syncthreads();
    // stage K [key][dim] and V^T [dim][key] (zeros past the prompt)
    for (int e = threadIdx.x; e < KB * (HD / 8); e += nthr) {
      const int j = e / (HD / 8), c = e % (HD / 8);
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (k0 + j < P) {
        kv = *(const uint4 *)(kbase + (size_t)(k0 + j) * HD + c * 8);
        vv = *(const uint4 *)(vbase + (size_t)(k0 + j) * HD + c * 8);
      }
      *(uint4 *)&ks[j][c * 8] = kv;
      const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        vt[c * 8 + 2 * q][j] = (uint16_t)(w[q] & 0xffffu);
        vt[c * 8 + 2 * q + 1][j] = (uint16_t)(w[q] >> 16);
      }
    }
    __syncthreads();
    if (wave < G) {
      // S = Q K^T
      pf_f32x4 s[2][4];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) s[mt][nt] = pf_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KS; ++st) {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const pf_bf16x8 kb = __builtin_bit_cast(pf_bf16x8, *(const uint4 *)&ks[nt * 16 + r16][st * 32 + grp * 8]);
#pragma unroll
          for (int mt = 0; mt < 2; ++mt)
            s[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[mt][st], kb, s[mt][nt], 0, 0, 0);
        }
      }
      // online softmax: lane holds rows mt*16 + grp*4 + i, key nt*16 + r16
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = q0 + mt * 16 + grp * 4 + i;
          float mx = -INFINITY;
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) {
            const int key = k0 + nt * 16 + r16;
            float v = s[mt][nt][i] * a.scale;
            if (key > row || key >= P) v = -INFINITY;
            s[mt][nt][i] = v;
            mx = fmaxf(mx, v);
          }
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
          const float mnew = fmaxf(mrun[mt][i], mx);
          const float alpha = (mnew == -INFINITY) ? 1.f : expf(mrun[mt][i] - mnew);
          float sum = 0.f;
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) {
            const float p = (s[mt][nt][i] == -INFINITY) ? 0.f : expf(s[mt][nt][i] - mnew);
            s[mt][nt][i] = p;
            sum += p;
          }
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) sum += __shfl_xor(sum, off, 64);
          lrun[mt][i] = lrun[mt][i] * alpha + sum;
          mrun[mt][i] = mnew;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) o[mt][dt][i] *= alpha;
        }
      }
      // P (bf16) to this wave's LDS tile, then O += P V
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i) pt[wave][mt * 16 + grp * 4 + i][nt * 16 + r16] = pf_f2bf(s[mt][nt][i]);
    }
    __syncthreads();
    if (wave < G) {
#pragma unroll
      for (int st = 0; st < KB / 32; ++st) {
        pf_bf16x8 pa[2];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          pa[mt] = __builtin_bit_cast(pf_bf16x8, *(const uint4 *)&pt[wave][mt * 16 + r16][st * 32 + grp * 8]);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const pf_bf16x8 vb = __builtin_bit_cast(pf_bf16x8, *(const uint4 *)&vt[dt * 16 + r16][st * 32 + grp * 8]);
#pragma unroll
          for (int mt = 0; mt < 2; ++mt) o[mt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[mt], vb, o[mt][dt], 0, 0, 0);
        }
      }
    }
  }
  if (wave >= G) return;
  // O / l -> bf16; lane holds rows mt*16 + grp*4 + i, dim dt*16 + r16
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = q0 + mt * 16 + grp * 4 + i;
      if (row >= P) continue;
      uint16_t *dst = (uint16_t *)a.out + (row_base + row) * a.ld_out + h * HD;
      const float inv = 1.f / lrun[mt][i];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) dst[dt * 16 + r16] = pf_f2bf(o[mt][dt][i] * inv);
    }
}

// ------------------------------------------------------------------------
// Decode attention on the matrix cores (bf16 caches, head_dim 64 or 128): one
// wave per work item (attn_mfma_item in attn_decode.h).
template <int HD>
__global__ __launch_bounds__(64) void attn_mfma_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t vr[ATT_SPLIT][HD + 16];
  __shared__ int prow[ATT_MAX_PAIRS];
  __shared__ int ppos[ATT_MAX_PAIRS];
  attn_mfma_item<HD>(a, blockIdx.x, blockIdx.y, vr, prow, ppos);
}

// The arguments of segment sg alone: its layer of the cache, its queries,
// rows and row groups, and the split records of its rows in the launch's
// row space (records of element type T).
template <typename T>
static __host__ __device__ inline void attn_seg_view(AttnArgs &a, const AttnSeg &sg) {
  const size_t r0 = (size_t)sg.r0;
  a.kc = sg.kc;
  a.vc = sg.vc;
  a.q += r0 * a.ldq;
  a.row_pos += r0;
  a.row_nc += r0;
  a.row_chain_off += r0;
  a.row_seq += r0;
  a.grp_row0 += sg.g0;
  a.grp_nrows += sg.g0;
  a.grp_seq += sg.g0;
  if (a.grp_nc != nullptr) a.grp_nc += sg.g0;
  a.n_rows = sg.M;
  a.n_splits = sg.n_splits;
  a.part = (T *)a.part + r0 * a.n_heads * a.jmax * a.head_dim;
  a.stat += r0 * a.n_heads * a.jmax * 2;
}

// Grouped form: block x runs item x - item0 of the segment whose items hold it.
template <int HD>
__global__ __launch_bounds__(64) void attn_mfma_seg_kernel(AttnArgs a, AttnSegs g) {
  __shared__ __attribute__((aligned(16))) uint16_t vr[ATT_SPLIT][HD + 16];
  __shared__ int prow[ATT_MAX_PAIRS];
  __shared__ int ppos[ATT_MAX_PAIRS];
  const int x = blockIdx.x;
  int k = 0;
#pragma unroll
  for (int i = 1; i < MAX_SEGS; ++i) k += (i < g.n && x >= g.item0[i]) ? 1 : 0;
  attn_seg_view<bf16>(a, g.s[k]);
  attn_mfma_item<HD>(a, x - g.item0[k], blockIdx.y, vr, prow, ppos);
}

// Causal prompt attention for head_dim 128 (bf16), G query heads per kv
// head with G in {1, 2, 4, 8}.  Workgroup = (32 query rows, kv head,
// sequence), wave w = query head kvh * G + w; blocks of 64 keys stream into
// a two-slot LDS ring with direct global -> LDS transfers (one block ahead of
// the products), shared by the G waves.  Per block each wave computes
//   S^T = K Q^T   four 16-key tiles against its two 16-query tiles, so each
//                 lane holds 16 keys of one query: the online-softmax
//                 statistics are that lane's plus an xor butterfly over the
//                 four quarter-waves, and the rescaling of O needs no
//                 exchange;
//   O^T += V^T P^T  V^T through the LDS transpose read, P^T straight from
//                 the S^T accumulators (k-slot e of a lane is key
//                 32 st + 4 grp + e or 32 st + 16 + 4 grp + e - 4, the keys it
//                 holds), O^T rows = head dims, columns = queries.
// K and V rows are 256 bytes with their 16-byte chunks XOR-swizzled (K: by
// row mod 16, V: by 2 (row mod 8)) so that the 16 rows of a K fragment read
// and the four rows of a transpose read land in distinct banks.  Query
// blocks are dispatched longest first (the causal triangle).
__device__ uint4 pa_zero[64];   // source of the key rows past the prompt

template <int G>
__global__ __launch_bounds__(64 * G) __attribute__((amdgpu_waves_per_eu(2))) void prefill_attn128_kernel(PrefillAttnArgs a) {
  constexpr int HD = 128, KS = 4, DT = 8, NKT = 4, QB = 32, KB = 64;
  constexpr int NTR = 2 * KB * HD * 2 / 1024;      // 1 KB transfers per key block (K then V)
  constexpr int PER_WAVE = NTR / G;
  __shared__ __attribute__((aligned(16))) uint4 kl[2][KB * 16];
  __shared__ __attribute__((aligned(16))) uint4 vl[2][KB * 16];

  const int P = a.prompt_len;
  const int nqb = (P + QB - 1) / QB;
  const int qb = nqb - 1 - (int)blockIdx.x;
  const int kvh = blockIdx.y, seq = blockIdx.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int tq = lane >> 4, ti = (lane & 15) >> 2, tg = lane & 3;
  const int h = kvh * G + wave;
  const int q0 = qb * QB;
  const size_t row_base = (size_t)seq * P;
  const uint16_t *kbase = (const uint16_t *)a.kc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;
  const uint16_t *vbase = (const uint16_t *)a.vc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;
  const int nblk = (min(q0 + QB, P) - 1) / KB + 1;

  // key block j into ring slot `slot`: transfer c (0..15 K, 16..31 V) moves
  // rows 4 (c mod 16) .. +3; lane l fills chunk position l mod 16 of row
  // 4 (c mod 16) + l / 16 with the swizzled global chunk
  const uintptr_t zero = (uintptr_t)(pa_zero + lane);
  auto issue = [&](int j, int slot) {
#pragma unroll
    for (int t = 0; t < PER_WAVE; ++t) {
      const int c = wave + G * t;
      const bool isv = c >= NTR / 2;
      const int ci = c % (NTR / 2);
      const int row = ci * 4 + (lane >> 4), pos = lane & 15;
      const int chunk = isv ? (pos ^ (2 * (row & 7))) : (pos ^ (row & 15));
      const int key = j * KB + row;
      const uintptr_t g = (uintptr_t)((isv ? vbase : kbase) + (size_t)key * HD + chunk * 8);
      const uintptr_t src = key < P ? g : zero;
      uint4 *dst = isv ? &vl[slot][ci * 64] : &kl[slot][ci * 64];
      __builtin_amdgcn_global_load_lds((const void *)src, (__attribute__((address_space(3))) void *)dst, 16, 0, 0);
    }
  };

  // Q^T fragments (B operand): lane (query r16 of tile mt, grp) holds dims
  // 32 st + 8 grp .. +8, rounded to bf16
  pf_bf16x8 qf[2][KS];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    const int row = q0 + mt * 16 + r16;
    const bool ok = row < P;
    const float *src = a.q + (row_base + (ok ? row : 0)) * a.ldq + h * HD + grp * 8;
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
      if (ok) {
        x0 = *(const float4 *)(src + st * 32);
        x1 = *(const float4 *)(src + st * 32 + 4);
      }
      qf[mt][st] = __builtin_bit_cast(pf_bf16x8, make_uint4(pf_pack_bf16(x0.x, x0.y), pf_pack_bf16(x0.z, x0.w),
                                                            pf_pack_bf16(x1.x, x1.y), pf_pack_bf16(x1.z, x1.w)));
    }
  }
  pf_f32x4 o[2][DT];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[mt][dt] = pf_f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun[2] = {-INFINITY, -INFINITY}, lrun[2] = {0.f, 0.f};
  const float sl2 = a.scale * 1.44269504088896341f;   // scores in log2 units

  issue(0, 0);
  for (int j = 0; j < nblk; ++j) {
    const int slot = j & 1, k0 = j * KB;
    lds_ring_step<0>();                      // block j has landed for every wave, and every
                                             // wave is past block j - 1
    if (j + 1 < nblk) issue(j + 1, slot ^ 1);
    const uint4 *K = kl[slot];
    // S^T = K Q^T
    pf_f32x4 sc[NKT][2];
#pragma unroll
    for (int nt = 0; nt < NKT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) sc[nt][mt] = pf_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KS; ++st)
#pragma unroll
      for (int nt = 0; nt < NKT; ++nt) {
        const pf_bf16x8 kfr = __builtin_bit_cast(pf_bf16x8, K[(nt * 16 + r16) * 16 + ((st * 4 + grp) ^ r16)]);
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          sc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kfr, qf[mt][st], sc[nt][mt], 0, 0, 0);
      }
    // online softmax of query q0 + 16 mt + r16 over keys k0 + 16 nt + 4 grp + i
    const bool diag = k0 + KB - 1 > q0;
    pf_bf16x8 pb[2][KB / 32];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int query = q0 + mt * 16 + r16;
      float mx = -INFINITY;
#pragma unroll
      for (int nt = 0; nt < NKT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = sc[nt][mt][i] * sl2;
          if (diag && k0 + nt * 16 + grp * 4 + i > query) v = -INFINITY;
          sc[nt][mt][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(mrun[mt], mx);
      const float mref = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(mrun[mt] - mref);
      float sum = 0.f;
#pragma unroll
      for (int nt = 0; nt < NKT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = __builtin_amdgcn_exp2f(sc[nt][mt][i] - mref);
          sc[nt][mt][i] = p;
          sum += p;
        }
      sum += __shfl_xor(sum, 16, 64);
      sum += __shfl_xor(sum, 32, 64);
      lrun[mt] = lrun[mt] * alpha + sum;
      mrun[mt] = mnew;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[mt][dt] *= alpha;
#pragma unroll
      for (int st = 0; st < KB / 32; ++st)
        pb[mt][st] = __builtin_bit_cast(
            pf_bf16x8, make_uint4(pf_pack_bf16(sc[2 * st][mt][0], sc[2 * st][mt][1]),
                                  pf_pack_bf16(sc[2 * st][mt][2], sc[2 * st][mt][3]),
                                  pf_pack_bf16(sc[2 * st + 1][mt][0], sc[2 * st + 1][mt][1]),
                                  pf_pack_bf16(sc[2 * st + 1][mt][2], sc[2 * st + 1][mt][3])));
    }
    // O^T += V^T P^T
    const uint16_t *V = (const uint16_t *)vl[slot];
#pragma unroll
    for (int st = 0; st < KB / 32; ++st) {
      const int rlo = 32 * st + 4 * tq + ti, rhi = rlo + 16;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int c = 2 * dt + (tg >> 1);
        const pf_bf16x8 vfr = tr_frag(V + (rlo * 16 + (c ^ (2 * (rlo & 7)))) * 8 + (tg & 1) * 4,
                                      V + (rhi * 16 + (c ^ (2 * (rhi & 7)))) * 8 + (tg & 1) * 4);
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          o[mt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vfr, pb[mt][st], o[mt][dt], 0, 0, 0);
      }
    }
  }
  // O / l -> bf16: lane holds dims 16 dt + 4 grp .. +3 of query q0 + 16 mt + r16
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    const int query = q0 + mt * 16 + r16;
    if (query >= P) continue;
    const float inv = 1.f / lrun[mt];
    uint16_t *dst = (uint16_t *)a.out + (row_base + query) * a.ld_out + h * HD + grp * 4;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *(uint2 *)(dst + dt * 16) = make_uint2(pf_pack_bf16(o[mt][dt][0] * inv, o[mt][dt][1] * inv),
                                             pf_pack_bf16(o[mt][dt][2] * inv, o[mt][dt][3] * inv));
  }
}

hipError_t launch_prefill_attention(const PrefillAttnArgs &a, hipStream_t s) {
  const int G = a.n_heads / a.n_kv_heads;
  if (G < 1 || G > 8 || a.prompt_len < 1) return hipErrorInvalidValue;
  dim3 grid((a.prompt_len + 31) / 32, a.n_kv_heads, a.batch);
  dim3 block(64 * G);
  if (a.head_dim == 128 && (G == 1 || G == 2 || G == 4 || G == 8) && a.ld_out % 4 == 0) {
    switch (G) {
      case 1: hipLaunchKernelGGL(prefill_attn128_kernel<1>, grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL(prefill_attn128_kernel<2>, grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL(prefill_attn128_kernel<4>, grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL(prefill_attn128_kernel<8>, grid, block, 0, s, a); break;
    }
    return hipGetLastError();
  }
  switch (a.head_dim) {
    case 64: hipLaunchKernelGGL(prefill_attn_kernel<64>, grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL(prefill_attn_kernel<128>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnArgs &a, int n_groups, hipStream_t s) {
  if (n_groups <= 0 || a.n_heads / a.n_kv_heads > 8) return hipErrorInvalidValue;
  if (a.n_splits < 1 || a.n_splits > a.jmax) return hipErrorInvalidValue;
  dim3 grid(n_groups, a.n_kv_heads, a.n_splits);
  if (dtype == 1 && (a.head_dim == 128 || a.head_dim == 64)) {
    if (a.n_rows < 1 || a.row_seq == nullptr) return hipErrorInvalidValue;
    const size_t items = 2 * (size_t)a.n_rows + (size_t)n_groups * a.n_splits;
    if (items > 0x7fffffffull) return hipErrorInvalidValue;
    dim3 g2((unsigned)items, a.n_kv_heads);
    if (a.head_dim == 128) hipLaunchKernelGGL(attn_mfma_kernel<128>, g2, dim3(64), 0, s, a);
    else hipLaunchKernelGGL(attn_mfma_kernel<64>, g2, dim3(64), 0, s, a);
    return hipGetLastError();
  }
  return dtype == 1 ? launch_attn_t<bf16>(a, grid, s) : launch_attn_t<float>(a, grid, s);
}

// The matrix-core kernel: up to MAX_SEGS segments per launch, a lone segment
// as a plain launch; the other kernels: one launch per segment.
hipError_t launch_attention_seg(int dtype, const AttnArgs &a, const AttnSeg *segs, int n, hipStream_t s) {
  if (segs == nullptr || n < 1 || a.n_heads / a.n_kv_heads > 8) return hipErrorInvalidValue;
  for (int i = 0; i < n; ++i) {
    const AttnSeg &sg = segs[i];
    if (sg.M < 1 || sg.r0 < 0 || sg.g0 < 0 || sg.n_groups < 1 || sg.n_splits < 1 || sg.n_splits > a.jmax)
      return hipErrorInvalidValue;
  }
  if (!(dtype == 1 && (a.head_dim == 128 || a.head_dim == 64))) {
    for (int i = 0; i < n; ++i) {
      AttnArgs b = a;
      if (dtype == 1) attn_seg_view<bf16>(b, segs[i]);
      else attn_seg_view<float>(b, segs[i]);
      const hipError_t e = launch_attention(dtype, b, segs[i].n_groups, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  if (a.row_seq == nullptr) return hipErrorInvalidValue;
  for (int i0 = 0; i0 < n; i0 += MAX_SEGS) {
    const int c = n - i0 < MAX_SEGS ? n - i0 : MAX_SEGS;
    if (c == 1) {
      AttnArgs b = a;
      attn_seg_view<bf16>(b, segs[i0]);
      const hipError_t e = launch_attention(1, b, segs[i0].n_groups, s);
      if (e != hipSuccess) return e;
      continue;
    }
    AttnSegs g{};
    g.n = c;
    size_t items = 0;
    for (int i = 0; i < c; ++i) {
      const AttnSeg &sg = segs[i0 + i];
      g.s[i] = sg;
      g.item0[i] = (int)items;
      items += 2 * (size_t)sg.M + (size_t)sg.n_groups * sg.n_splits;
      if (items > 0x7fffffffull) return hipErrorInvalidValue;
    }
    for (int i = c; i < MAX_SEGS; ++i) g.item0[i] = (int)items;
    const dim3 grid((unsigned)items, a.n_kv_heads);
    if (a.head_dim == 128) hipLaunchKernelGGL(attn_mfma_seg_kernel<128>, grid, dim3(64), 0, s, a, g);
    else hipLaunchKernelGGL(attn_mfma_seg_kernel<64>, grid, dim3(64), 0, s, a, g);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace dex
