// Internal declarations shared by the HIP kernels and the host engine.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dex {

// Output column of local tile row r16 (0..15) of QKV tile `tile`: a tile keeps
// the two RoPE partners (i, i + hd/2) of one head together -- rows 0..7 are
// dims 8j..8j+7 and rows 8..15 dims hd/2+8j.. of head tile/(hd/16), j the
// tile's index inside the head.  Shared by weight packing and the epilogues.
__device__ __forceinline__ int qkv_col(int tile, int r16, int hd) {
  const int tph = hd / 16;                 // tiles per head
  const int head = tile / tph, j = tile % tph;
  const int dim = (r16 < 8) ? (8 * j + r16) : (hd / 2 + 8 * j + r16 - 8);
  return head * hd + dim;
}

typedef uint16_t bf16;

// Step of an LDS ring filled by direct global -> LDS transfers
// (global_load_lds): wait until at most VMCNT of this wave's vector-memory
// operations are outstanding (the oldest transfers have landed in LDS), then
// meet the workgroup's other waves.  Unlike __syncthreads() it does not wait
// for the younger transfers still in flight.  The empty asm statements emit
// nothing; they keep the compiler from moving any memory access across the
// wait and the barrier.
template <int VMCNT>
__device__ __forceinline__ void lds_ring_step() {
  static_assert(VMCNT >= 0 && VMCNT < 16, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70 | VMCNT);   // lgkmcnt, expcnt: no wait
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Sampling-mode Gumbel noise of token v for the slot of sequence `seq` at
// position `pos` (the definition is stated with dex_debug_gumbel in dex.h).
__device__ __forceinline__ unsigned long long sm64_mix(unsigned long long z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
__device__ __forceinline__ unsigned long long gumbel_key(unsigned long long seed, int seq, int pos) {
  return sm64_mix(seed ^ sm64_mix(((unsigned long long)(unsigned)seq << 32) + (unsigned long long)(unsigned)pos));
}
__device__ __forceinline__ float gumbel_noise(unsigned long long key, int v) {
  const unsigned long long z = sm64_mix(key + (unsigned long long)(v + 1) * 0x9E3779B97F4A7C15ull);
  const float u = ((float)(unsigned)(z >> 41) + 0.5f) * (1.0f / 8388608.0f);
  return -logf(-logf(u));
}

// ---------------------------------------------------------------- epilogues
enum Epi {
  EPI_PLAIN = 0,   // y[m][n] (float)
  EPI_QKV = 1,     // rms-scaled, RoPE on q/k, q -> float buffer, k/v -> cache
  EPI_RESID = 2,   // h += alpha * y; next-norm input and sum-of-squares partials
  EPI_SWIGLU = 3,  // rms-scaled gate/up pair -> SiLU(gate) * up
  EPI_LOGITS = 4,  // rms-scaled LM head, DECS mask, per-tile argmax
  EPI_BIAS_SILU = 5,  // SiLU(rms-scaled y + bias) -> act (adapter up-projection)
};

constexpr int GEMM_WAVES = 8;       // split-K ways inside a workgroup
constexpr int GEMM_THREADS = GEMM_WAVES * 64;
constexpr int ATT_SPLIT = 64;       // logical keys per attention split (one wave)
constexpr int ATT_THREADS = 64;
constexpr int ATT_MAX_PAIRS = 64;   // (row, query head) pairs per attention row group
constexpr int ATT_MAX_SPLITS = 4096; // longest context: 262144 positions

struct GemmArgs {
  // Weights in the packed block layout (see PackArgs); nsteps_w k-steps per tile.
  const void *wp;
  int nsteps_w;
  int N;          // output columns (SWIGLU: d_ffn)
  int K;
  const void *x;  // activations [M][ldx]
  int ldx;
  int M;
  // RMSNorm scale from sum-of-squares partials (nullable): per row
  // 1/sqrt(sum(part[m][0..n_part)) * inv_d + eps).
  const float *part;
  int n_part;
  float inv_d, eps;
  // Prompt GEMMs (launch_gemm_tiled): the same scales precomputed per row by
  // launch_row_scale, required there whenever part is set.
  const float *row_rsc;
  // PLAIN / QKV: float output [M][ld_out]
  float *out;
  int ld_out;
  // QKV
  void *kc, *vc;              // this layer's cache base ([B][Hkv][E][hd])
  int kv_entries;             // E
  int n_heads, n_kv_heads, head_dim;
  const int *row_seq, *row_pos, *row_entry;
  const float2 *rope;         // [max_ctx][hd/2] (cos, sin)
  // RESID
  float *h;                   // [M][ld_h] residual stream (in place)
  int ld_h;
  float alpha;
  const float *g_next;        // gain of the next RMSNorm (nullable)
  void *xb;                   // next-norm input g*h (T) [M][ld_h] (nullable)
  float *part_out;            // [M][n_part_out]
  int n_part_out;
  const int *row_bnd;         // nullable: write h/partials to boundary storage instead
  float *bnd_h, *bnd_part;
  const float *bias;          // RESID (nullable): h += alpha * (y + bias); BIAS_SILU: SiLU(y + bias)
  // SWIGLU
  void *act;                  // [M][ld_act] (T)
  int ld_act;
  // LOGITS
  const int *mask_tok;        // [M][mask_stride]
  const int *mask_n;          // [M]
  int mask_stride;
  float *logits_tap;          // nullable [M][N]
  float2 *amax;               // [M][n_tiles] (value, index as float bits)
  int n_tiles;
  float temperature;          // > 0: Gumbel-max sampling with the rows of (sample_seed, row_seq, row_pos)
  unsigned long long sample_seed;
};

// Split partials of R rows live in one buffer of R * H * jmax * (hd + 2)
// floats: the split outputs o in the cache's element type ([R][H][jmax][hd],
// filling at most the first R * H * jmax * hd floats), then the statistics
// ([R][H][jmax] of float (max, sum)) at float offset R * H * jmax * hd.
inline float *split_stats(float *part, size_t rows, int n_heads, int jmax, int hd) {
  return part + rows * n_heads * jmax * hd;
}

struct AttnArgs {
  const float *q;             // [R][H*hd], RoPE applied
  int ldq;
  const void *kc, *vc;        // this layer's cache base
  int kv_entries, n_kv_heads, n_heads, head_dim, batch;
  // row groups: consecutive rows of one sequence that share their committed
  // prefix; grp_nc (nullable) is that prefix's length
  const int *grp_row0, *grp_nrows, *grp_seq, *grp_nc;
  const int *row_pos, *row_nc, *row_chain_off, *chain;
  const int *row_seq;         // sequence of each row (matrix-core kernel)
  int n_rows;                 // rows of the launch (matrix-core kernel)
  void *part;                 // [R][H][jmax][hd] split outputs o (element type of the cache)
  float *stat;                // [R][H][jmax][2] their (max, sum)
  int jmax;                   // split stride of `part` and `stat`
  int n_splits;               // splits the launch covers: max over its rows of pos / 64 + 1 (<= jmax)
  float scale;
};

struct CombineArgs {
  const void *part;           // as AttnArgs
  const float *stat;
  const int *row_pos;
  int jmax, n_heads, head_dim;
  void *out;                  // [R][H*hd] (T)
  int ld_out;
};

// Grouped launches.  The stages of a round are independent and, taken in
// step, all run their j-th layer at the same time: one launch then covers
// that layer step of every stage (a segment each), each segment on its own
// rows of the launch's row space with its own layer's weights and cache.  A
// segment's rows go through exactly the arithmetic of a launch of their own
// (segments never share a workgroup), so grouping changes no result bit.
// A launch takes at most MAX_SEGS segments in its arguments (longer lists go
// out as several launches), and a single segment goes out as a plain launch
// of the same rows: the arguments stay small, which keeps the launch cost of
// short kernels down.
constexpr int MAX_SEGS = 8;

struct GemmSeg {
  const void *wp;             // the segment's layer weights (packed)
  void *kc, *vc;              // QKV: the layer's key/value cache base
  const float *g_next;        // RESID: the next RMSNorm's gain (nullptr: none)
  const int *row_bnd;         // RESID: boundary rows of the segment (nullable)
  float alpha;                // RESID: the layer's residual scale
  int r0, M;                  // rows [r0, r0 + M) of the launch's buffers
};
struct GemmSegs {
  int n;
  GemmSeg s[MAX_SEGS];
};

// The arguments of segment s alone: its weights and layer, and the
// row-indexed buffers and tables advanced to its first row.
template <typename T, int EPI>
__host__ __device__ inline void gemm_seg_view(GemmArgs &a, const GemmSeg &s) {
  static_assert(EPI == EPI_QKV || EPI == EPI_RESID || EPI == EPI_SWIGLU, "grouped epilogues");
  const size_t r = (size_t)s.r0;
  a.wp = s.wp;
  a.M = s.M;
  a.x = (const T *)a.x + r * a.ldx;
  if (a.part != nullptr) a.part += r * a.n_part;
  if constexpr (EPI == EPI_QKV) {
    a.out += r * a.ld_out;
    a.kc = s.kc;
    a.vc = s.vc;
    a.row_seq += r;
    a.row_pos += r;
    a.row_entry += r;
  } else if constexpr (EPI == EPI_RESID) {
    a.h += r * a.ld_h;
    a.alpha = s.alpha;
    a.g_next = s.g_next;
    a.xb = s.g_next != nullptr ? (void *)((T *)a.xb + r * a.ld_h) : nullptr;
    a.part_out += r * a.n_part_out;
    a.row_bnd = s.row_bnd;
  } else {
    a.act = (T *)a.act + r * a.ld_act;
  }
}

struct AttnSeg {
  const void *kc, *vc;        // the segment's layer of the cache
  int r0, M;                  // its rows [r0, r0 + M) of the queries and row tables
  int g0, n_groups;           // its row groups [g0, g0 + n_groups) (row0 relative to r0)
  int n_splits;               // 64-key splits up to its deepest row
};
struct AttnSegs {
  int n;
  int item0[MAX_SEGS];        // first work item of each segment (set by the launcher)
  AttnSeg s[MAX_SEGS];
};

// Causal prompt attention on the matrix cores (bf16 keys/values, head_dim 64
// or 128): rows are (sequence, position) in order, keys are the committed
// cache entries 0..position.
struct PrefillAttnArgs {
  const float *q;             // [batch * prompt_len][ldq], RoPE applied
  int ldq;
  const void *kc, *vc;        // this layer's cache base
  int kv_entries, n_kv_heads, n_heads, head_dim, batch, prompt_len;
  float scale;
  void *out;                  // [batch * prompt_len][ld_out] (bf16)
  int ld_out;
};
hipError_t launch_prefill_attention(const PrefillAttnArgs &a, hipStream_t s);

// Weight packing.  mode 0: rows in order; 1: QKV, the three segments w0/w1/w2
// concatenated with each tile holding RoPE partner dimensions (i, i + hd/2)
// of one head; 2: gate (w0) and up (w1) blocks interleaved per step.
struct PackArgs {
  const void *w0, *w1, *w2;
  int n0, n1, n2;
  int N, K, mode, head_dim;
  void *out;
  int nsteps;     // filled by launch_pack
};
size_t packed_bytes(int dtype, int N, int K, int mode);
hipError_t launch_pack(int dtype, const PackArgs &a, hipStream_t s);

// Launchers (return the HIP status of the launch).
hipError_t launch_gemm(int dtype, int epi, const GemmArgs &a, int m_blocks, hipStream_t s);
// Prompt-prefill GEMM (bf16, M-tiled: 128 weight rows x 128 input rows per
// workgroup) with the QKV / RESID / SWIGLU / PLAIN epilogues.  Requires N a
// multiple of 16, K a multiple of 8, 16-byte aligned rows and no boundary
// rows (gemm_tiled_supported); launch_gemm_tiled returns hipErrorInvalidValue
// otherwise.  A normed GEMM takes its row scales from row_rsc.
bool gemm_tiled_supported(int epi, const GemmArgs &a);
hipError_t launch_gemm_tiled(int epi, const GemmArgs &a, hipStream_t s);
// out[m] = 1 / sqrt(sum(part[m][0..n_part)) * inv_d + eps), m < M: the RMSNorm
// scales launch_gemm_tiled reads, summed in index order.
hipError_t launch_row_scale(const float *part, int n_part, int M, float inv_d, float eps, float *out, hipStream_t s);
hipError_t launch_attention(int dtype, const AttnArgs &a, int n_groups, hipStream_t s);
hipError_t launch_combine(int dtype, const CombineArgs &a, int rows, hipStream_t s);
// Grouped forms (QKV, RESID and SWIGLU epilogues; the decode attention):
// `a` holds what the segments share, with the row-indexed buffers and tables
// at row 0 of the launch.  The attention's split records then use the row
// space of the launch: part [rows][H][jmax][hd], stat at split_stats(part,
// rows, ...), where rows covers every segment.
hipError_t launch_gemm_seg(int dtype, int epi, const GemmArgs &a, const GemmSeg *segs, int n, hipStream_t s);
hipError_t launch_attention_seg(int dtype, const AttnArgs &a, const AttnSeg *segs, int n, hipStream_t s);

struct PrepArgs {
  int M, d, n_part;
  int embed_rows;             // rows [0, embed_rows): h = E[token]; the others h = boundary[src]
  const int *row_tok;         // embed token per row
  const int *row_src;         // boundary index per row
  const void *embed;
  const float *bnd_h, *bnd_part;
  const float *g;             // gain of the first RMSNorm the rows meet
  // n_seg > 0: segments of consecutive rows (one per stage of a grouped
  // lane), rows [seg_end[k-1], seg_end[k]) meeting gain seg_g[k] instead of g
  int n_seg;
  int seg_end[MAX_SEGS];
  const float *seg_g[MAX_SEGS];
  float *h, *part;            // [M][d], [M][n_part]
  void *xb;                   // [M][d] (T)
  const int *row_out;         // nullable: write h/part to row_out[m] instead of m
};
hipError_t launch_prep(int dtype, const PrepArgs &a, hipStream_t s);

struct ArgmaxArgs {
  const float2 *amax;
  int n_tiles, M;
  int *u_out;                 // [M]
  int *cand;                  // [..][N] candidate table (nullable)
  const int *row_cand;        // [M] index into cand (slot*N + stage)
  // verify/commit of the rows that complete an anchor's final stage
  // (nullable): row_commit[m] = i >= 0 writes (token, k*) to commit_out[2i..]
  const int *row_commit;
  int N;
  int *commit_out;
};
hipError_t launch_argmax(const ArgmaxArgs &a, hipStream_t s);

struct CollapseArgs {
  int n_jobs;
  const int *job;             // [n_jobs][6]: seq, src entry, dst entry, src slot, dst slot, kind (0 kv only, 1 kv + slot state)
  void *kc, *vc;              // cache base
  int n_layers, batch, n_kv_heads, kv_entries, head_dim;
  int elem_bytes;
  float *bnd_h, *bnd_part;    // [B][2S][d], [B][2S][n_part]
  int *cand;                  // [B][2S][N]
  int slots2, d, n_part, N, max_ctx, S;
};
hipError_t launch_collapse(const CollapseArgs &a, hipStream_t s);

hipError_t launch_gumbel(unsigned long long seed, int seq, int pos, int V, float *out, hipStream_t s);
hipError_t launch_copy(void *dst, const void *src, int64_t bytes, hipStream_t s);

}  // namespace dex
