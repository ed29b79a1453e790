// M-tiled matrix-core GEMM for the prompt prefill on gfx950 (bf16).
//
//   acc[m][n] = sum_k x[m][k] * W[n][k]
//
// With M = batch x prompt length in the tens of thousands the skinny decode
// kernel would re-read the activations once per 16-column weight tile; here a
// workgroup of four waves owns 128 weight rows x 128 input rows and each wave
// a 64 x 64 block of 4 x 4 v_mfma_f32_16x16x32_bf16 tiles (the gate/up pair:
// 2 tile pairs x 4).  Both operands come straight from memory in fragment
// order: the packed weight layout stores one MFMA A fragment of a 16-row tile
// per 1 KB block, and an input fragment is 16 rows x 64 contiguous bytes.
// Neighbouring waves share operands through L1/L2.  The next k-step is loaded
// while the current one is multiplied.  When its grid reaches 96 workgroups,
// a second form (gemm_big_kernel) stages the operands through LDS in
// 256 x 256 workgroup tiles; it computes every output element from the same
// MFMA operands in the same order, so the two forms give the same bits.
//
// The epilogues are those of the decode kernel (RMSNorm row scale, RoPE and
// the key/value cache write; residual add with the next norm's input and its
// sum-of-squares partials; SwiGLU), applied to the accumulators in registers:
// lane (g, r) of a tile holds output rows 4g..4g+3 of input row r, so every
// store covers four consecutive columns.  The row scales of a normed GEMM
// are computed once beforehand (row_scale_kernel) rather than by each of
// its column blocks.
#include "dex_kernels.h"

namespace dex {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 tb_bf16x8;
typedef __attribute__((ext_vector_type(4))) float tb_f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int tb_u32x4;

constexpr int TB_THREADS = 256;   // 2 x 2 waves
constexpr int TB_MF = 4;          // 16-row input fragments per wave (64 rows)
constexpr int TB_ROWS = 128;      // input rows per workgroup

__device__ __forceinline__ uint32_t tb_f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ uint2 tb_pack4(float a, float b, float c, float d) {
  return make_uint2(tb_f2bf(a) | (tb_f2bf(b) << 16), tb_f2bf(c) | (tb_f2bf(d) << 16));
}

// Sum of a row's n sum-of-squares partials in index order.  The loads go out
// 32 at a time, so that a batch waits for one memory latency rather than
// one per partial; the padding terms are +0, which leaves the sum (>= +0)
// unchanged.
__device__ __forceinline__ float tb_part_sum(const float *p, int n) {
  float ss = 0.f;
  for (int q0 = 0; q0 < n; q0 += 32) {
    float v[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) v[i] = q0 + i < n ? p[q0 + i] : 0.f;
#pragma unroll
    for (int i = 0; i < 32; ++i) ss += v[i];
  }
  return ss;
}

// RMSNorm reciprocal scale of every prompt row, once per normed GEMM (each
// of a GEMM's column blocks would otherwise reduce the row's partials
// again): one thread per row.
__global__ __launch_bounds__(256) void row_scale_kernel(const float *part, int n_part, int M, float inv_d, float eps,
                                                        float *out) {
  const int m = blockIdx.x * 256 + threadIdx.x;
  if (m >= M) return;
  const float ss = tb_part_sum(part + (size_t)m * n_part, n_part);
  out[m] = 1.0f / sqrtf(ss * inv_d + eps);
}

// Epilogue of one 16 x 16 output tile held by a wave: lane (g, r) holds
// output columns tile*16 + 4g .. +3 of input row m (ok: m < M).  Every lane
// of the wave calls it (the RESID form exchanges values across lanes).
// acc[0] is the tile (SwiGLU: the gate tile, acc[1] the up tile), rsc the
// row's RMSNorm scale.  The QKV epilogue is tb_qkv_block.
template <int EPI, int NT>
__device__ __forceinline__ void tb_epilogue(const GemmArgs &a, int tile, int m, bool ok, const tb_f32x4 (&acc)[NT],
                                            float rsc, int grp) {
  if constexpr (EPI == EPI_PLAIN) {
    if (ok) {
      float *o = a.out + (size_t)m * a.ld_out + tile * 16 + grp * 4;
      *(float4 *)o = make_float4(acc[0][0], acc[0][1], acc[0][2], acc[0][3]);
    }
  } else if constexpr (EPI == EPI_RESID) {
    const int n0 = tile * 16 + grp * 4;
    float hn[4] = {0.f, 0.f, 0.f, 0.f};
    if (ok) {
      float *hp = a.h + (size_t)m * a.ld_h + n0;
      const float4 hv = *(const float4 *)hp;
      hn[0] = hv.x + a.alpha * acc[0][0];
      hn[1] = hv.y + a.alpha * acc[0][1];
      hn[2] = hv.z + a.alpha * acc[0][2];
      hn[3] = hv.w + a.alpha * acc[0][3];
      *(float4 *)hp = make_float4(hn[0], hn[1], hn[2], hn[3]);
      if (a.xb != nullptr) {
        const float *gn = a.g_next + n0;
        *(uint2 *)((uint16_t *)a.xb + (size_t)m * a.ld_h + n0) =
            tb_pack4(gn[0] * hn[0], gn[1] * hn[1], gn[2] * hn[2], gn[3] * hn[3]);
      }
    }
    // sum of squares over the tile's 16 columns: four per lane, then
    // across the four lane groups that hold the same input row
    float sq = hn[0] * hn[0] + hn[1] * hn[1] + hn[2] * hn[2] + hn[3] * hn[3];
    sq += __shfl_xor(sq, 16, 64);
    sq += __shfl_xor(sq, 32, 64);
    if (ok && grp == 0) a.part_out[(size_t)m * a.n_part_out + tile] = sq;
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (ok) {
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float gt = acc[0][i] * rsc, up = acc[NT - 1][i] * rsc;
        o[i] = gt / (1.0f + expf(-gt)) * up;
      }
      *(uint2 *)((uint16_t *)a.act + (size_t)m * a.ld_act + tile * 16 + grp * 4) = tb_pack4(o[0], o[1], o[2], o[3]);
    }
  }
}

// QKV epilogue of the tiles T0 .. T0 + NTL - 1 (consecutive) over NF input
// fragments (lane (g, r) of fragment f: input row mbase + 16 f + r): RMSNorm
// scale, RoPE on the query and key columns (the tile's rows 0..7 hold
// dimensions i of a head, rows 8..15 dimensions i + hd/2: the partner of a
// value sits 32 lanes away), queries to out (fp32), keys and values to the
// cache entry of the row.  The row-table loads, and the RoPE-table loads of
// four tiles at a time, are issued before the stores they feed, so that
// they are not held behind stores to memory the compiler cannot tell apart
// from the tables.
template <int NTL, int NF, typename Acc>
__device__ __forceinline__ void tb_qkv_block(const GemmArgs &a, int T0, int mbase, const float (&rsc)[NF], int r16,
                                             int grp, Acc acc) {
  const int hd = a.head_dim;
  const int nq = a.n_heads * hd, nk = a.n_kv_heads * hd;
  const int n_tiles = a.N / 16;
  const bool lo = grp < 2;
  int pos[NF], seq[NF], ent[NF];
  bool ok[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int m = mbase + f * 16 + r16;
    ok[f] = m < a.M;
    const int mm = ok[f] ? m : 0;
    pos[f] = a.row_pos[mm];
    seq[f] = a.row_seq[mm];
    ent[f] = a.row_entry[mm];
  }
  constexpr int CH = NTL < 4 ? NTL : 4;     // tiles per batch of RoPE loads
  static_assert(NTL % CH == 0, "tile batches");
#pragma unroll
  for (int f = 0; f < NF; ++f) {
#pragma unroll
    for (int p0 = 0; p0 < NTL; p0 += CH) {
      float4 cs[CH][2];                        // (cos, sin) of the lane's four pairs
#pragma unroll
      for (int q = 0; q < CH; ++q) {
        const int p = p0 + q, tile = T0 + p;
        const int col0 = qkv_col(tile, 0, hd), head_col = col0 - col0 % hd;
        const int i0 = 8 * (tile % (hd / 16)) + (grp & 1) * 4;
        if (tile < n_tiles && head_col < nq + nk) {
          const float4 *rp = (const float4 *)(a.rope + (size_t)pos[f] * (hd / 2) + i0);
          cs[q][0] = rp[0];
          cs[q][1] = rp[1];
        } else {
          cs[q][0] = cs[q][1] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int q = 0; q < CH; ++q) {
        const int p = p0 + q, tile = T0 + p;
        if (tile >= n_tiles) continue;         // uniform across the wave
        const int col0 = qkv_col(tile, 0, hd), head_col = col0 - col0 % hd;
        const int i0 = 8 * (tile % (hd / 16)) + (grp & 1) * 4;
        const tb_f32x4 t = acc(p, f);
        const float c[4] = {cs[q][0].x, cs[q][0].z, cs[q][1].x, cs[q][1].z};
        const float sn[4] = {cs[q][0].y, cs[q][0].w, cs[q][1].y, cs[q][1].w};
        float y[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = t[i] * rsc[f];
          const float partner = __shfl_xor(v, 32, 64);
          y[i] = v;
          if (ok[f] && head_col < nq + nk)     // q or k: rotate the pair
            y[i] = lo ? v * c[i] - partner * sn[i] : v * c[i] + partner * sn[i];
        }
        if (!ok[f]) continue;
        const int dim0 = (lo ? 0 : hd / 2) + i0;
        if (head_col < nq) {
          *(float4 *)(a.out + (size_t)(mbase + f * 16 + r16) * a.ld_out + head_col + dim0) =
              make_float4(y[0], y[1], y[2], y[3]);
        } else {
          const bool isk = head_col < nq + nk;
          const int g = (isk ? head_col - nq : head_col - nq - nk) / hd;
          uint16_t *cache = (uint16_t *)(isk ? a.kc : a.vc);
          const size_t base = (((size_t)seq[f] * a.n_kv_heads + g) * a.kv_entries + ent[f]) * hd;
          *(uint2 *)(cache + base + dim0) = tb_pack4(y[0], y[1], y[2], y[3]);
        }
      }
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(TB_THREADS) void gemm_tiled_kernel(GemmArgs a) {
  constexpr int NT = (EPI == EPI_SWIGLU) ? 2 : 1;   // interleaved gate/up blocks
  constexpr int TN = 4 / NT;                        // weight tiles per wave
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int n_tiles = a.N / 16;
  const int tile0 = (blockIdx.x * 2 + (wave & 1)) * TN;
  const int m_base = blockIdx.y * TB_ROWS + (wave >> 1) * 64;
  const int nsteps = a.nsteps_w;

  const char *wp[TN];
  bool tok[TN];
#pragma unroll
  for (int t = 0; t < TN; ++t) {
    tok[t] = tile0 + t < n_tiles;
    wp[t] = (const char *)a.wp + (size_t)(tok[t] ? tile0 + t : 0) * nsteps * NT * 1024 + lane * 16;
  }
  const uint16_t *xr[TB_MF];
  bool xok[TB_MF];
#pragma unroll
  for (int f = 0; f < TB_MF; ++f) {
    const int m = m_base + f * 16 + r16;
    xok[f] = m < a.M;
    xr[f] = (const uint16_t *)a.x + (size_t)(xok[f] ? m : 0) * a.ldx + grp * 8;
  }

  tb_f32x4 acc[TN][NT][TB_MF];
#pragma unroll
  for (int t = 0; t < TN; ++t)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int f = 0; f < TB_MF; ++f) acc[t][nt][f] = tb_f32x4{0.f, 0.f, 0.f, 0.f};

  tb_u32x4 wa[TN][NT], xa[TB_MF], wb[TN][NT], xb[TB_MF];
  auto load = [&](int s, tb_u32x4 (&w)[TN][NT], tb_u32x4 (&x)[TB_MF]) {
    const bool sin = s < nsteps;
    const bool kin = sin && (s * 32 + grp * 8 < a.K);
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        w[t][nt] = (sin && tok[t]) ? *(const tb_u32x4 *)(wp[t] + ((size_t)s * NT + nt) * 1024)
                                   : tb_u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int f = 0; f < TB_MF; ++f)
      x[f] = (kin && xok[f]) ? *(const tb_u32x4 *)(xr[f] + s * 32) : tb_u32x4{0u, 0u, 0u, 0u};
  };
  auto mma = [&](const tb_u32x4 (&w)[TN][NT], const tb_u32x4 (&x)[TB_MF]) {
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int f = 0; f < TB_MF; ++f)
          acc[t][nt][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(tb_bf16x8, w[t][nt]), __builtin_bit_cast(tb_bf16x8, x[f]), acc[t][nt][f], 0, 0, 0);
  };
  load(0, wa, xa);
  for (int s = 0; s < nsteps; s += 2) {
    load(s + 1, wb, xb);
    mma(wa, xa);
    if (s + 1 >= nsteps) break;
    load(s + 2, wa, xa);
    mma(wb, xb);
  }

  // RMSNorm scale of each input row (lane j sums the partials of row
  // m_base + j in order), then handed to the lanes holding that row
  float rsc[TB_MF];
#pragma unroll
  for (int f = 0; f < TB_MF; ++f) {
    const int m = m_base + f * 16 + r16;
    rsc[f] = (a.row_rsc != nullptr && m < a.M) ? a.row_rsc[m] : 1.f;
  }

  if constexpr (EPI == EPI_QKV) {
    tb_qkv_block<TN, TB_MF>(a, tile0, m_base, rsc, r16, grp, [&](int t, int f) { return acc[t][0][f]; });
  } else {
#pragma unroll
    for (int t = 0; t < TN; ++t) {
      if (!tok[t]) continue;                  // uniform across the wave
#pragma unroll
      for (int f = 0; f < TB_MF; ++f) {
        const int m = m_base + f * 16 + r16;
        tb_f32x4 at[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) at[nt] = acc[t][nt][f];
        tb_epilogue<EPI, NT>(a, tile0 + t, m, m < a.M, at, rsc[f], grp);
      }
    }
  }
}

// Large form, taken whenever its grid has at least BG_MIN_WG workgroups
// (below that the 128 x 128 form keeps more CUs busy).  A workgroup of eight
// waves owns 256 weight rows (16 packed blocks per k-step: 16 tiles, or 8
// gate/up pairs) x 256 input rows and stages both operands through LDS in
// fragment order, so each operand byte fetched from L2 feeds 16 MFMA tiles
// instead of 2.  The k-steps (32 KB each) move global -> LDS with direct
// transfers (global_load_lds, 16 bytes per lane at LDS base + 16 x lane)
// into a ring of four slots, three steps ahead of the products: no staging
// registers, and each wave waits (vmcnt) only for its own oldest step before
// the per-step barrier.  Wave (wn, wm) multiplies weight blocks
// 8 wn .. 8 wn + 7 by input fragments 4 wm .. 4 wm + 3 (128 x 64 outputs)
// with the operand roles of gemm_tiled_kernel, accumulating the k-steps in
// order, and hands each tile to the shared epilogue.  Workgroups are
// numbered so that each XCD takes a contiguous run of tiles, grouped eight
// input blocks deep, which keeps the operands the XCD's waves share in its
// own L2.
constexpr int BG_THREADS = 512;
constexpr int BG_ROWS = 256;      // input rows per workgroup
constexpr int BG_BLK = 16;        // weight blocks per k-step per workgroup
constexpr int BG_NBUF = 4;        // LDS stages in the ring (three in flight)
constexpr int BG_GROUP = 8;       // input blocks per tile group
constexpr int BG_MIN_WG = 96;     // smallest grid that takes this form

__device__ tb_u32x4 bg_zero[64];  // source of the zero lanes outside the operands

#define BG_LDS(p) ((__attribute__((address_space(3))) void *)(p))

template <int EPI>
__global__ __launch_bounds__(BG_THREADS) void gemm_big_kernel(GemmArgs a, int n_blk_n, int n_wg) {
  constexpr int NT = (EPI == EPI_SWIGLU) ? 2 : 1;   // interleaved gate/up blocks
  constexpr int TPW = BG_BLK / NT;                  // output tiles per workgroup
  constexpr int WB = 8;                             // weight blocks per wave
  constexpr int WF = 4;                             // input fragments per wave
  constexpr int NBLK = 2 * BG_BLK;                  // 1 KB blocks per stage
  __shared__ tb_u32x4 lds[BG_NBUF][NBLK][64];       // [stage slot][weight blocks | fragments][lane]

  const int xcd = blockIdx.x % 8, jx = blockIdx.x / 8;
  const int base = n_wg / 8, rem = n_wg % 8;
  const int t = xcd * base + min(xcd, rem) + jx;
  const int n_blk_m = n_wg / n_blk_n;
  const int per_group = BG_GROUP * n_blk_n;
  const int g = t / per_group, first_m = g * BG_GROUP;
  const int gsize = min(BG_GROUP, n_blk_m - first_m);
  const int mb = first_m + (t % per_group) % gsize, nb = (t % per_group) / gsize;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int wn = wave & 1, wm = wave >> 1;
  const int n_tiles = a.N / 16, nsteps = a.nsteps_w;
  const int tile0 = nb * TPW, m0 = mb * BG_ROWS;

  tb_f32x4 acc[WB][WF];
#pragma unroll
  for (int jb = 0; jb < WB; ++jb)
#pragma unroll
    for (int f = 0; f < WF; ++f) acc[jb][f] = tb_f32x4{0.f, 0.f, 0.f, 0.f};

  // one k-step into slot `slot`: wave w moves weight blocks w, w + 8 and
  // input fragments w, w + 8 (1 KB each) global -> LDS, one instruction per
  // block; lanes outside the operands read zeros.  The source is chosen by
  // selects, so every wave issues exactly NBLK / 8 transfers per step.
  const uintptr_t zero = (uintptr_t)(bg_zero + lane);
  auto issue = [&](int step, int slot) {
#pragma unroll
    for (int i = 0; i < NBLK / 8; ++i) {
      const int b = wave + 8 * i;
      uintptr_t src;
      if (i < 2) {                            // weight block b
        const int tile = tile0 + b / NT, nt = b % NT;
        const uintptr_t wa = (uintptr_t)a.wp + (((size_t)tile * nsteps + step) * NT + nt) * 1024 + lane * 16;
        src = tile < n_tiles ? wa : zero;
      } else {                                // input fragment b - 16
        const int m = m0 + (b - BG_BLK) * 16 + r16, k = step * 32 + grp * 8;
        const uintptr_t xa = (uintptr_t)((const uint16_t *)a.x + (size_t)m * a.ldx + k);
        src = ((m < a.M) & (k < a.K)) ? xa : zero;
      }
      __builtin_amdgcn_global_load_lds((const void *)src, BG_LDS(&lds[slot][b][0]), 16, 0, 0);
    }
  };
  for (int s = 0; s < BG_NBUF - 1 && s < nsteps; ++s) issue(s, s);
  for (int st = 0; st < nsteps; ++st) {
    // this wave's transfers of step st are done once at most those of the
    // (up to two) younger steps are outstanding; the barrier makes every
    // wave's done, and tells that all waves have finished step st - 1
    const int younger = min(nsteps - 1 - st, BG_NBUF - 2);
    if (younger >= 2) lds_ring_step<8>();
    else if (younger == 1) lds_ring_step<4>();
    else lds_ring_step<0>();
    if (st + BG_NBUF - 1 < nsteps) issue(st + BG_NBUF - 1, (st + BG_NBUF - 1) % BG_NBUF);
    const int slot = st % BG_NBUF;
    tb_u32x4 w[WB], x[WF];
#pragma unroll
    for (int jb = 0; jb < WB; ++jb) w[jb] = lds[slot][wn * WB + jb][lane];
#pragma unroll
    for (int f = 0; f < WF; ++f) x[f] = lds[slot][BG_BLK + wm * WF + f][lane];
#pragma unroll
    for (int jb = 0; jb < WB; ++jb)
#pragma unroll
      for (int f = 0; f < WF; ++f)
        acc[jb][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(tb_bf16x8, w[jb]),
                                                             __builtin_bit_cast(tb_bf16x8, x[f]), acc[jb][f], 0, 0, 0);
  }

  // RMSNorm scale of each input row of the wave (lane j sums the partials of
  // row m0 + 64 wm + j in order), handed to the lanes holding that row
  float rsc[WF];
#pragma unroll
  for (int f = 0; f < WF; ++f) {
    const int m = m0 + wm * 64 + f * 16 + r16;
    rsc[f] = (a.row_rsc != nullptr && m < a.M) ? a.row_rsc[m] : 1.f;
  }
  if constexpr (EPI == EPI_QKV) {
    tb_qkv_block<WB, WF>(a, tile0 + wn * WB, m0 + wm * 64, rsc, r16, grp, [&](int p, int f) { return acc[p][f]; });
  } else {
#pragma unroll
    for (int p = 0; p < WB / NT; ++p) {
      const int tile = tile0 + wn * (WB / NT) + p;
      if (tile >= n_tiles) continue;          // uniform across the wave
#pragma unroll
      for (int f = 0; f < WF; ++f) {
        const int m = m0 + wm * 64 + f * 16 + r16;
        tb_f32x4 at[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) at[nt] = acc[p * NT + nt][f];
        tb_epilogue<EPI, NT>(a, tile, m, m < a.M, at, rsc[f], grp);
      }
    }
  }
}

}  // namespace

bool gemm_tiled_supported(int epi, const GemmArgs &a) {
  if (a.M < 1 || a.N < 16 || a.N % 16 || a.K < 8 || a.K % 8 || a.ldx % 8 || a.row_bnd != nullptr) return false;
  if (a.part != nullptr && a.row_rsc == nullptr) return false;   // the row scales come precomputed
  if ((a.M + TB_ROWS - 1) / TB_ROWS > 65535) return false;
  switch (epi) {
    case EPI_PLAIN: return a.ld_out % 4 == 0;
    case EPI_QKV: return a.ld_out % 4 == 0 && a.head_dim % 16 == 0;
    case EPI_RESID: return a.ld_h % 4 == 0;
    case EPI_SWIGLU: return a.ld_act % 4 == 0;
    default: return false;
  }
}

hipError_t launch_row_scale(const float *part, int n_part, int M, float inv_d, float eps, float *out, hipStream_t s) {
  if (part == nullptr || out == nullptr || n_part < 1 || M < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(row_scale_kernel, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, part, n_part, M, inv_d, eps,
                     out);
  return hipGetLastError();
}

hipError_t launch_gemm_tiled(int epi, const GemmArgs &a, hipStream_t s) {
  if (!gemm_tiled_supported(epi, a)) return hipErrorInvalidValue;
  const int n_tiles = a.N / 16;
  const int tpw = BG_BLK / (epi == EPI_SWIGLU ? 2 : 1);
  const int n_blk_n = (n_tiles + tpw - 1) / tpw, n_blk_m = (a.M + BG_ROWS - 1) / BG_ROWS;
  const long long n_wg = (long long)n_blk_n * n_blk_m;
  if (n_wg >= BG_MIN_WG) {
    if (n_wg > 0x7fffffffLL) return hipErrorInvalidValue;
    dim3 grid((unsigned)n_wg), block(BG_THREADS);
    switch (epi) {
      case EPI_PLAIN: hipLaunchKernelGGL(gemm_big_kernel<EPI_PLAIN>, grid, block, 0, s, a, n_blk_n, (int)n_wg); break;
      case EPI_QKV: hipLaunchKernelGGL(gemm_big_kernel<EPI_QKV>, grid, block, 0, s, a, n_blk_n, (int)n_wg); break;
      case EPI_RESID: hipLaunchKernelGGL(gemm_big_kernel<EPI_RESID>, grid, block, 0, s, a, n_blk_n, (int)n_wg); break;
      case EPI_SWIGLU: hipLaunchKernelGGL(gemm_big_kernel<EPI_SWIGLU>, grid, block, 0, s, a, n_blk_n, (int)n_wg); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int tiles_per_wg = epi == EPI_SWIGLU ? 4 : 8;
  dim3 grid((n_tiles + tiles_per_wg - 1) / tiles_per_wg, (a.M + TB_ROWS - 1) / TB_ROWS);
  dim3 block(TB_THREADS);
  switch (epi) {
    case EPI_PLAIN: hipLaunchKernelGGL(gemm_tiled_kernel<EPI_PLAIN>, grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL(gemm_tiled_kernel<EPI_QKV>, grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL(gemm_tiled_kernel<EPI_RESID>, grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL(gemm_tiled_kernel<EPI_SWIGLU>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dex
