// Skinny-M matrix-core GEMM for the decode step on gfx950.
//
//   acc[m][n] = sum_k x[m][k] * W[n][k]          (W row-major [N][K])
//
// The M <= 64 rows of a round are tiny next to the weights, so the kernel is
// a weight stream: one workgroup owns a 16-column tile of W (two tiles for
// the gate/up pair), its eight waves split K by interleaved 16-byte steps,
// and each wave issues 128-bit loads of W (A operand, 16 rows x 64 bytes per
// instruction) and of x (B operand, from L2) into v_mfma_f32_16x16x32_bf16
// (bf16) or v_mfma_f32_16x16x4_f32 (fp32) tiles.  Rows beyond M are zero.
// The split-K partials meet in LDS and are summed in wave order, so a row's
// result depends only on its own input: the same bits for any M, any
// neighbouring rows and any position in the batch.
//
// Epilogues fuse the elementwise work of a transformer layer:
//   QKV     RMSNorm scale (from the producer's sum-of-squares partials), RoPE
//           on q and k, q to a float buffer, k and v to the key/value cache
//           at each row's entry;
//   RESID   h += alpha * acc, the next RMSNorm's input g*h in the matrix-core
//           type, and per-16-column sum-of-squares partials of h;
//   SWIGLU  SiLU(r*gate) * (r*up) for the interleaved gate/up tiles;
//   BIAS_SILU  SiLU(r*acc + bias) (the inducing adapter's first layer);
//   RESID with a bias: h += alpha * (acc + bias) (its second layer);
//   LOGITS  r*acc, optional float logits tap, in sampling mode acc/tau plus
//           the slot's Gumbel noise, DECS mask (-inf), and the tile's argmax
//           (lowest id on ties);
//   PLAIN   float output (tests).
#include "gemm_common.h"

namespace dex {

// U: k-steps per prefetch chunk (two chunks in flight per wave).  It only
// sets how far loads run ahead: every wave still accumulates its steps in
// increasing order, so the result does not depend on U.  NTW: weight tiles
// per workgroup; with many rows a second tile halves the activation loads
// per weight byte.  A tile's sums are the same per-wave partials added in
// the same order whatever NTW is, so neither changes any result bit.
template <typename T, int EPI, int MB, int U, int NTW>
__device__ __forceinline__ void gemm_tile(const GemmArgs &a) {
  using F = Frag<T>;
  constexpr int EPB = F::EPB;
  constexpr int KSTEP = 4 * EPB;               // k covered by one 16-byte step of a wave
  constexpr int NT = (EPI == EPI_SWIGLU) ? 2 : 1;
  constexpr int NA = NT * NTW;                 // weight blocks per step of the workgroup
  __shared__ float red_all[NA][GEMM_WAVES][MB][64][4];
  __shared__ float val[NA][16][16 * MB];
  __shared__ float rs[16 * MB];

  const int tile0 = blockIdx.x * NTW;
  const int n_tiles = (a.N + 15) / 16;
  const int m0 = blockIdx.y * 16 * MB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int Mloc = min(16 * MB, a.M - m0);

  // ---- this lane's weight streams: packed 1 KB blocks, one per (tile, step, t)
  const char *wbase[NTW];
  bool wok[NTW];
#pragma unroll
  for (int tw = 0; tw < NTW; ++tw) {
    wok[tw] = tile0 + tw < n_tiles;
    wbase[tw] = (const char *)a.wp + (size_t)(wok[tw] ? tile0 + tw : 0) * a.nsteps_w * NT * 1024 + lane * 16;
  }
  // ---- this lane's activation rows (one per M block)
  const T *xrow[MB];
  bool xok[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + mb * 16 + r16;
    xok[mb] = m < a.M;
    xrow[mb] = (const T *)a.x + (size_t)(xok[mb] ? m : 0) * a.ldx;
  }

  f32x4_t acc[NA][MB];
#pragma unroll
  for (int t = 0; t < NA; ++t)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[t][mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nsteps = a.nsteps_w;
  F wa[U][NA], xa[U][MB], wb[U][NA], xb[U][MB];

  auto load_chunk = [&](int s0, F (&w)[U][NA], F (&x)[U][MB]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int s = s0 + u * GEMM_WAVES;
      const int k = s * KSTEP + grp * EPB;
      const bool kin = (s < nsteps) && (k < a.K);
#pragma unroll
      for (int tw = 0; tw < NTW; ++tw)
#pragma unroll
        for (int t = 0; t < NT; ++t)
          w[u][tw * NT + t].v = load16(wbase[tw] + ((size_t)s * NT + t) * 1024, s < nsteps && wok[tw]);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) x[u][mb].v = load16_cached(xrow[mb] + k, kin && xok[mb]);
    }
  };
  auto compute_chunk = [&](const F (&w)[U][NA], const F (&x)[U][MB]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < NA; ++t)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[t][mb] = F::mma(w[u][t], x[u][mb], acc[t][mb]);
  };

  int s = wave;
  const int stride = U * GEMM_WAVES;
  if (s < nsteps) load_chunk(s, wa, xa);
  while (s < nsteps) {
    const int sn = s + stride;
    if (sn < nsteps) load_chunk(sn, wb, xb);
    compute_chunk(wa, xa);
    s = sn;
    if (s >= nsteps) break;
    const int sn2 = s + stride;
    if (sn2 < nsteps) load_chunk(sn2, wa, xa);
    compute_chunk(wb, xb);
    s = sn2;
  }

  // ---- split-K partials meet in LDS, summed in wave order
#pragma unroll
  for (int t = 0; t < NA; ++t)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red_all[t][wave][mb][lane][i] = acc[t][mb][i];

  // RMSNorm scales of this block's rows
  if (a.part != nullptr) {
    for (int ml = wave; ml < Mloc; ml += GEMM_WAVES) {
      const float r = row_rscale(a.part + (size_t)(m0 + ml) * a.n_part, a.n_part, a.inv_d, a.eps, lane);
      if (lane == 0) rs[ml] = r;
    }
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < NA; ++t) reduce_block<MB>(red_all[t], val[t]);
  __syncthreads();

  // ---- epilogues, one weight tile at a time
  for (int tw = 0; tw < NTW; ++tw) {
  const int tile = tile0 + tw;
  if (tile >= n_tiles) break;
  float (*vt)[16][16 * MB] = &val[tw * NT];
  if constexpr (EPI == EPI_PLAIN) {
    for (int e = threadIdx.x; e < 16 * Mloc; e += GEMM_THREADS) {
      const int ml = e / 16, nl = e % 16;
      const int n = tile * 16 + nl;
      if (n < a.N) a.out[(size_t)(m0 + ml) * a.ld_out + n] = vt[0][nl][ml];
    }
  } else if constexpr (EPI == EPI_QKV) {
    const int hd = a.head_dim;
    const int col0 = qkv_col(tile, 0, hd);       // first column of the tile
    const int nq = a.n_heads * hd, nk = a.n_kv_heads * hd;
    const int j = tile % (hd / 16);
    for (int e = threadIdx.x; e < 8 * Mloc; e += GEMM_THREADS) {
      const int ml = e / 8, p = e % 8;           // pair p: dims 8j+p and hd/2+8j+p
      const int m = m0 + ml;
      const float r = (a.part != nullptr) ? rs[ml] : 1.f;
      float x1 = vt[0][p][ml] * r, x2 = vt[0][p + 8][ml] * r;
      const int i = 8 * j + p;
      const int c1 = col0 - (col0 % hd) + i;    // column of dim i in this head
      const int c2 = c1 + hd / 2;
      if (c1 < nq + nk) {                        // q or k: rotate
        const float2 cs = a.rope[(size_t)a.row_pos[m] * (hd / 2) + i];
        const float y1 = x1 * cs.x - x2 * cs.y;
        const float y2 = x2 * cs.x + x1 * cs.y;
        x1 = y1;
        x2 = y2;
      }
      if (c1 < nq) {
        a.out[(size_t)m * a.ld_out + c1] = x1;
        a.out[(size_t)m * a.ld_out + c2] = x2;
      } else {
        const bool isk = c1 < nq + nk;
        const int cc = isk ? c1 - nq : c1 - nq - nk;
        const int g = cc / hd, dim = cc % hd;
        T *cache = (T *)(isk ? a.kc : a.vc);
        const size_t base = (((size_t)a.row_seq[m] * a.n_kv_heads + g) * a.kv_entries + a.row_entry[m]) * hd;
        cache[base + dim] = to_t<T>(x1);
        cache[base + dim + hd / 2] = to_t<T>(x2);
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    __shared__ float sq[16][16 * MB];
    epi_resid<T, MB>(a, tile, m0, Mloc, vt[0], sq);
  } else if constexpr (EPI == EPI_SWIGLU) {
    for (int e = threadIdx.x; e < 16 * Mloc; e += GEMM_THREADS) {
      const int ml = e / 16, nl = e % 16;
      const int m = m0 + ml, n = tile * 16 + nl;
      if (n >= a.N) continue;
      const float r = (a.part != nullptr) ? rs[ml] : 1.f;
      const float gt = vt[0][nl][ml] * r, up = vt[NT - 1][nl][ml] * r;
      const float sg = gt / (1.0f + expf(-gt));
      ((T *)a.act)[(size_t)m * a.ld_act + n] = to_t<T>(sg * up);
    }
  } else if constexpr (EPI == EPI_BIAS_SILU) {
    for (int e = threadIdx.x; e < 16 * Mloc; e += GEMM_THREADS) {
      const int ml = e / 16, nl = e % 16;
      const int m = m0 + ml, n = tile * 16 + nl;
      if (n >= a.N) continue;
      const float r = (a.part != nullptr) ? rs[ml] : 1.f;
      const float u = vt[0][nl][ml] * r + a.bias[n];
      ((T *)a.act)[(size_t)m * a.ld_act + n] = to_t<T>(u / (1.0f + expf(-u)));
    }
  } else if constexpr (EPI == EPI_LOGITS) {
    __shared__ float z[16][16 * MB];
    for (int e = threadIdx.x; e < 16 * Mloc; e += GEMM_THREADS) {
      const int ml = e / 16, nl = e % 16;
      const int m = m0 + ml, n = tile * 16 + nl;
      const float r = (a.part != nullptr) ? rs[ml] : 1.f;
      float v = vt[0][nl][ml] * r;
      if (n < a.N) {
        if (a.logits_tap != nullptr) a.logits_tap[(size_t)m * a.N + n] = v;
        // sampling mode (Algorithm 2): the Gumbel row of the row's slot
        if (a.temperature > 0.f)
          v = v / a.temperature + gumbel_noise(gumbel_key(a.sample_seed, a.row_seq[m], a.row_pos[m]), n);
      } else {
        v = -INFINITY;
      }
      z[nl][ml] = v;
    }
    __syncthreads();
    // DECS mask: each (row, masked token) pair clears its column if the token
    // falls in this tile (one pass, every table load issued at once)
    for (int e = threadIdx.x; e < Mloc * a.mask_stride; e += GEMM_THREADS) {
      const int ml = e / a.mask_stride, q = e % a.mask_stride;
      const int m = m0 + ml;
      if (q < a.mask_n[m]) {
        const int nn = a.mask_tok[(size_t)m * a.mask_stride + q] - tile * 16;
        if (nn >= 0 && nn < 16) z[nn][ml] = -INFINITY;
      }
    }
    __syncthreads();
    for (int ml = threadIdx.x; ml < Mloc; ml += GEMM_THREADS) {
      float best = -INFINITY;
      int bi = -1;
#pragma unroll
      for (int nl = 0; nl < 16; ++nl) {
        const float v = z[nl][ml];
        if (v > best || bi < 0) { best = v; bi = tile * 16 + nl; }
      }
      a.amax[(size_t)(m0 + ml) * a.n_tiles + tile] = make_float2(best, __int_as_float(bi));
    }
  }
  __syncthreads();                             // epilogue scratch is reused by the next tile
  }
}

template <typename T, int EPI, int MB, int U, int NTW>
__global__ __launch_bounds__(GEMM_THREADS) void gemm_kernel(GemmArgs a) {
  gemm_tile<T, EPI, MB, U, NTW>(a);
}

// Segment blockIdx.z of a grouped launch (gemm_seg_view); row blocks past
// its rows have nothing to do.
template <typename T, int EPI, int MB, int U, int NTW>
__global__ __launch_bounds__(GEMM_THREADS) void gemm_seg_kernel(GemmArgs a, GemmSegs g) {
  gemm_seg_view<T, EPI>(a, g.s[blockIdx.z]);
  if ((int)blockIdx.y * 16 * MB >= a.M) return;
  gemm_tile<T, EPI, MB, U, NTW>(a);
}

// Weight packing: block (tile, step, t) holds, for lane l, the 16 bytes of
// row col(tile, l % 16) at k = step * KSTEP + (l / 16) * EPB (zeros beyond
// N or K), so that a wave's load of one MFMA step is one contiguous 1 KB.
template <typename T>
__global__ __launch_bounds__(64) void pack_kernel(PackArgs a) {
  constexpr int EPB = 16 / (int)sizeof(T);
  constexpr int KSTEP = 4 * EPB;
  const int NT = a.mode == 2 ? 2 : 1;
  const size_t blk = blockIdx.x;
  const int t = (int)(blk % NT);
  const size_t ts = blk / NT;
  const int step = (int)(ts % a.nsteps);
  const int tile = (int)(ts / a.nsteps);
  const int lane = threadIdx.x, r16 = lane & 15, grp = lane >> 4;
  const int col = (a.mode == 1) ? qkv_col(tile, r16, a.head_dim) : tile * 16 + r16;
  const int k = step * KSTEP + grp * EPB;
  u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
  if (col < a.N && k < a.K) {
    const T *base;
    int r;
    if (a.mode == 2) { base = (const T *)(t == 0 ? a.w0 : a.w1); r = col; }
    else if (col < a.n0) { base = (const T *)a.w0; r = col; }
    else if (col < a.n0 + a.n1) { base = (const T *)a.w1; r = col - a.n0; }
    else { base = (const T *)a.w2; r = col - a.n0 - a.n1; }
    v = *(const u32x4_t *)(base + (size_t)r * a.K + k);
  }
  *((u32x4_t *)((char *)a.out + blk * 1024) + lane) = v;
}

size_t packed_bytes(int dtype, int N, int K, int mode) {
  const int kstep = dtype == 1 ? 32 : 16;
  const size_t tiles = (N + 15) / 16, steps = (K + kstep - 1) / kstep;
  return tiles * steps * (mode == 2 ? 2 : 1) * 1024;
}

hipError_t launch_pack(int dtype, const PackArgs &a, hipStream_t s) {
  const int kstep = dtype == 1 ? 32 : 16;
  PackArgs b = a;
  b.nsteps = (a.K + kstep - 1) / kstep;
  const size_t blocks = (size_t)((a.N + 15) / 16) * b.nsteps * (a.mode == 2 ? 2 : 1);
  if (blocks == 0) return hipSuccess;
  if (dtype == 1) hipLaunchKernelGGL(pack_kernel<bf16>, dim3((unsigned)blocks), dim3(64), 0, s, b);
  else hipLaunchKernelGGL(pack_kernel<float>, dim3((unsigned)blocks), dim3(64), 0, s, b);
  return hipGetLastError();
}

// One launch of the chosen configuration: plain, or grouped over g's
// segments (grid z).
template <typename T, int EPI, int MB, int U, int NTW>
static void go(const GemmArgs &a, const GemmSegs *g, dim3 grid, hipStream_t s) {
  if constexpr (EPI == EPI_QKV || EPI == EPI_RESID || EPI == EPI_SWIGLU) {
    if (g != nullptr) {
      hipLaunchKernelGGL((gemm_seg_kernel<T, EPI, MB, U, NTW>), dim3(grid.x, grid.y, g->n), dim3(GEMM_THREADS), 0,
                         s, a, *g);
      return;
    }
  }
  hipLaunchKernelGGL((gemm_kernel<T, EPI, MB, U, NTW>), grid, dim3(GEMM_THREADS), 0, s, a);
}

// Weight tiles per workgroup of a projection with 256 (O, down) or 384 (QKV)
// tiles at up to 32 rows over nseg segments: every activation load feeds
// NTW tiles, which pays from 5 rows on once the grid still fills the chip;
// at 1-4 rows a grouped launch keeps one tile with a shallower prefetch
// (measured per class, row count and segment count on the 32-layer d4096
// model, lone QKV launches at 1-4 rows inside the decode step; 0: the
// general table).
static int proj_tiles_per_wg(int n_tiles, int M, int nseg) {
  if (M > 32 || n_tiles < 256 || n_tiles > 384) return 0;
  const bool qkv = n_tiles > 256;
  if (nseg == 1) return qkv && M > 4 ? 2 : 0;
  if (M <= 4) return 1;
  if (nseg == 2) return qkv ? 4 : 2;
  if (nseg <= 4) return qkv ? 2 : (nseg == 4 && M <= 8 ? 2 : 4);
  return 4;
}

// The configuration for M rows (a grouped launch of nseg segments: its
// largest segment's).
template <typename T, int EPI>
static hipError_t launch_t(const GemmArgs &a, const GemmSegs *g, int M, int nseg, hipStream_t s) {
  const int n_tiles = (a.N + 15) / 16;
  if constexpr (EPI == EPI_QKV || EPI == EPI_RESID) {
    const int ntw = proj_tiles_per_wg(n_tiles, M, nseg);
    if (ntw == 1) {
      go<T, EPI, 1, 2, 1>(a, g, dim3(n_tiles, 1), s);
      return hipGetLastError();
    }
    if (ntw > 0 && M <= 16) {
      if (ntw == 4) go<T, EPI, 1, 2, 4>(a, g, dim3((n_tiles + 3) / 4, 1), s);
      else if (nseg == 1) go<T, EPI, 1, 8, 2>(a, g, dim3((n_tiles + 1) / 2, 1), s);
      else go<T, EPI, 1, 4, 2>(a, g, dim3((n_tiles + 1) / 2, 1), s);
      return hipGetLastError();
    }
    if (ntw > 0) {
      if (ntw == 4) go<T, EPI, 2, 2, 4>(a, g, dim3((n_tiles + 3) / 4, 1), s);
      else if (EPI == EPI_QKV && nseg > 1) go<T, EPI, 2, 2, 2>(a, g, dim3((n_tiles + 1) / 2, 1), s);
      else go<T, EPI, 2, 4, 2>(a, g, dim3((n_tiles + 1) / 2, 1), s);
      return hipGetLastError();
    }
  }
  if (M <= 16) {
    // deeper prefetch when a workgroup per CU streams a long tile, shallower
    // when many workgroups share each CU (measured on the 4096-wide layers);
    // from 5 rows on, the wide matrices (gate/up, LM head) take two tiles per
    // workgroup so that each activation load feeds two weight tiles
    if (M > 4 && n_tiles > 512)
      go<T, EPI, 1, 2, 2>(a, g, dim3((n_tiles + 1) / 2, 1), s);
    else if (n_tiles <= 256) go<T, EPI, 1, 8, 1>(a, g, dim3(n_tiles, 1), s);
    else if (n_tiles <= 1024) go<T, EPI, 1, 4, 1>(a, g, dim3(n_tiles, 1), s);
    else go<T, EPI, 1, 2, 1>(a, g, dim3(n_tiles, 1), s);
  } else {
    // more rows: the wide matrices take several weight tiles per workgroup
    // so that each activation load feeds them all -- four for the 2000-tile
    // LM head and for gate/up up to 32 rows, two for gate/up beyond; the
    // 256-tile projections take two tiles per workgroup and split the rows
    // over a second grid row from 25 rows on (the same 256 workgroups, each
    // activation load feeding two tiles); the 384-tile QKV keeps one tile
    // per workgroup (measured per class at 17-64 rows); with 64-row blocks
    // the reduction buffer takes most of the LDS
    if (M <= 32) {
      if constexpr (EPI == EPI_LOGITS || EPI == EPI_SWIGLU)
        go<T, EPI, 2, 2, 4>(a, g, dim3((n_tiles + 3) / 4, 1), s);
      else if (n_tiles <= 256 && M > 24)
        go<T, EPI, 1, 8, 2>(a, g, dim3((n_tiles + 1) / 2, 2), s);
      else if (n_tiles <= 256)
        go<T, EPI, 2, 8, 1>(a, g, dim3(n_tiles, 1), s);
      else
        go<T, EPI, 2, 4, 1>(a, g, dim3(n_tiles, 1), s);
    } else if (n_tiles <= 256 && EPI != EPI_LOGITS && EPI != EPI_SWIGLU) {
      go<T, EPI, 2, 4, 2>(a, g, dim3((n_tiles + 1) / 2, (M + 31) / 32), s);
    } else {
      const unsigned mb = (unsigned)((M + 63) / 64);
      if constexpr (EPI == EPI_LOGITS)
        go<T, EPI, 4, 2, 4>(a, g, dim3((n_tiles + 3) / 4, mb), s);
      else if constexpr (EPI == EPI_SWIGLU)
        go<T, EPI, 4, 2, 2>(a, g, dim3((n_tiles + 1) / 2, mb), s);
      else
        go<T, EPI, 4, 4, 1>(a, g, dim3(n_tiles, mb), s);
    }
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, int epi, const GemmArgs &a, int m_blocks, hipStream_t s) {
  if (m_blocks <= 0) return hipErrorInvalidValue;
  if (dtype == 1) {
    switch (epi) {
      case EPI_PLAIN: return launch_t<bf16, EPI_PLAIN>(a, nullptr, a.M, 1, s);
      case EPI_QKV: return launch_t<bf16, EPI_QKV>(a, nullptr, a.M, 1, s);
      case EPI_RESID: return launch_t<bf16, EPI_RESID>(a, nullptr, a.M, 1, s);
      case EPI_SWIGLU: return launch_t<bf16, EPI_SWIGLU>(a, nullptr, a.M, 1, s);
      case EPI_LOGITS: return launch_t<bf16, EPI_LOGITS>(a, nullptr, a.M, 1, s);
      case EPI_BIAS_SILU: return launch_t<bf16, EPI_BIAS_SILU>(a, nullptr, a.M, 1, s);
    }
  } else {
    switch (epi) {
      case EPI_PLAIN: return launch_t<float, EPI_PLAIN>(a, nullptr, a.M, 1, s);
      case EPI_QKV: return launch_t<float, EPI_QKV>(a, nullptr, a.M, 1, s);
      case EPI_RESID: return launch_t<float, EPI_RESID>(a, nullptr, a.M, 1, s);
      case EPI_SWIGLU: return launch_t<float, EPI_SWIGLU>(a, nullptr, a.M, 1, s);
      case EPI_LOGITS: return launch_t<float, EPI_LOGITS>(a, nullptr, a.M, 1, s);
      case EPI_BIAS_SILU: return launch_t<float, EPI_BIAS_SILU>(a, nullptr, a.M, 1, s);
    }
  }
  return hipErrorInvalidValue;
}

// Up to MAX_SEGS segments per launch; a lone segment as a plain launch.
template <typename T, int EPI>
static hipError_t launch_seg_t(const GemmArgs &a, const GemmSeg *segs, int n, hipStream_t s) {
  for (int i0 = 0; i0 < n; i0 += MAX_SEGS) {
    const int c = n - i0 < MAX_SEGS ? n - i0 : MAX_SEGS;
    hipError_t e;
    if (c == 1) {
      GemmArgs b = a;
      gemm_seg_view<T, EPI>(b, segs[i0]);
      e = launch_t<T, EPI>(b, nullptr, b.M, 1, s);
    } else {
      GemmSegs g{};
      g.n = c;
      int M = 0;
      for (int i = 0; i < c; ++i) {
        g.s[i] = segs[i0 + i];
        M = g.s[i].M > M ? g.s[i].M : M;
      }
      e = launch_t<T, EPI>(a, &g, M, c, s);
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_gemm_seg(int dtype, int epi, const GemmArgs &a, const GemmSeg *segs, int n, hipStream_t s) {
  if (n < 1 || segs == nullptr) return hipErrorInvalidValue;
  for (int i = 0; i < n; ++i)
    if (segs[i].M < 1 || segs[i].r0 < 0) return hipErrorInvalidValue;
  if (dtype == 1) {
    switch (epi) {
      case EPI_QKV: return launch_seg_t<bf16, EPI_QKV>(a, segs, n, s);
      case EPI_RESID: return launch_seg_t<bf16, EPI_RESID>(a, segs, n, s);
      case EPI_SWIGLU: return launch_seg_t<bf16, EPI_SWIGLU>(a, segs, n, s);
    }
  } else {
    switch (epi) {
      case EPI_QKV: return launch_seg_t<float, EPI_QKV>(a, segs, n, s);
      case EPI_RESID: return launch_seg_t<float, EPI_RESID>(a, segs, n, s);
      case EPI_SWIGLU: return launch_seg_t<float, EPI_SWIGLU>(a, segs, n, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace dex
