/*
 * dex.h -- C ABI of the MI355X (gfx950) Depth Exploration Decoding library.
 *
 * One library context decodes `batch` independent sequences, each with its
 * own depth-position lattice, greedily, exactly as Algorithm 1 of the paper
 * ("Depth Exploration for LLM Decoding") describes:
 *   - dex_create    : a model with exit depths and an explored-depth set X
 *                     (Definition 3: d_0 < ... < d_{N-1} = L) go in;
 *                     stage k is the layer range (d_{k-1}, d_k] (Algorithm 1,
 *                     Require clause).
 *   - dex_prefill   : Algorithm 1's init -- the prompt's keys/values and the
 *                     first generated token (final-depth argmax at the last
 *                     prompt position).
 *   - dex_step      : one iteration of Algorithm 1's loop (expand, DECS,
 *                     insert, and when the anchor reaches the final depth
 *                     validate-and-commit then collapse) for every sequence;
 *                     commits at most one token per sequence.
 *   - dex_destroy   : frees everything the library allocated.
 *
 * The committed tokens equal greedy autoregressive decoding of the same
 * model (the lossless invariant of Section 3.2); with X = {L} and
 * width_cap = 1 each dex_step is one plain autoregressive step.
 *
 * Conventions
 *   - Every call returns dex_status; DEX_OK is 0, errors are negative.  No
 *     C++ exception crosses the ABI.  dex_last_error(ctx) gives a message
 *     (dex_last_error(NULL): the last dex_create failure of this thread).
 *   - Weights are passed as DEVICE memory, row-major; a projection matrix is
 *     [out_features][in_features].  dex_create repacks every projection
 *     matrix and the LM head into the library's own streaming layout, so a
 *     context holds a second, library-owned copy of those weights (one more
 *     model's worth of device memory: about 14.2 GB for a 32-layer d_model
 *     4096 model) until dex_destroy.  The caller's embedding table and norm
 *     gains stay borrowed: keep them alive and unchanged until dex_destroy
 *     (the caller's projection and LM-head arrays may be freed once
 *     dex_create has returned).  The library also owns the key/value caches,
 *     the lattice state and all scratch memory.
 *   - Host arrays passed in or out are caller-owned and only accessed during
 *     the call.
 *   - All device work is enqueued on config.hip_stream (NULL = the default
 *     stream).  dex_prefill and dex_step synchronise that stream before
 *     returning host results.  A context is not thread-safe.
 *   - Argument errors (DEX_E_INVAL), a prefill that could not allocate its
 *     scratch (DEX_E_NOMEM) and "every sequence is full" (DEX_E_CAPACITY
 *     before any work) leave the context as it was.  Any other failure
 *     inside an entry point -- a failed HIP call, a lattice capacity
 *     overflow found after the round's planning began, a host/device commit
 *     mismatch -- poisons it: later dex_prefill / dex_step calls return
 *     DEX_E_STATE; dex_destroy still frees everything.
 */
#ifndef DEX_H
#define DEX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dex_ctx dex_ctx;

typedef enum {
  DEX_OK = 0,
  DEX_E_INVAL = -1,     /* bad argument (dims, explored set, sizes, null pointers) */
  DEX_E_NOMEM = -2,     /* device or host allocation failed */
  DEX_E_HIP = -3,       /* a HIP runtime call failed; message in dex_last_error */
  DEX_E_STATE = -4,     /* call out of order (step before prefill) or poisoned context */
  DEX_E_CAPACITY = -5   /* max_context or lattice capacity exhausted */
} dex_status;

typedef enum { DEX_F32 = 0, DEX_BF16 = 1 } dex_dtype;

/* Per-layer parameter order inside dex_model.layers. */
enum {
  DEX_P_ATTN_NORM = 0,  /* float [d]                    RMSNorm gain before attention */
  DEX_P_WQ = 1,         /* weight [H*hd][d]             query projection */
  DEX_P_WK = 2,         /* weight [Hkv*hd][d]           key projection */
  DEX_P_WV = 3,         /* weight [Hkv*hd][d]           value projection */
  DEX_P_WO = 4,         /* weight [d][H*hd]             attention output projection */
  DEX_P_FFN_NORM = 5,   /* float [d]                    RMSNorm gain before the FFN */
  DEX_P_W_GATE = 6,     /* weight [F][d]                SwiGLU gate projection */
  DEX_P_W_UP = 7,       /* weight [F][d]                SwiGLU up projection */
  DEX_P_W_DOWN = 8,     /* weight [d][F]                SwiGLU down projection */
  DEX_P_COUNT = 9
};

#define DEX_MAX_BATCH 64
#define DEX_MAX_EXPLORED 32
#define DEX_MAX_ROWS 256

/* "A model with exit depths": a decoder-only Llama-family backbone whose
 * shared final RMSNorm and LM head decode every explored depth (the paper's
 * inducing-adapter appendix: intermediate depths use the same final
 * normalisation and LM head).  Layer l (1-based) scales both residual
 * branches by residual_scale * l / L.  RoPE is rotate-half with base
 * rope_theta; attention scale 1/sqrt(head_dim); query head h reads key/value
 * head h / (n_heads / n_kv_heads).  `weight_dtype` is the element type of the
 * embedding, the projections and the LM head, and also of the key/value
 * cache and the activations fed to the matrix cores; norm gains are float.
 * Requirements: d_model a multiple of 16; head_dim 32, 64 or 128; n_heads
 * a multiple of n_kv_heads; n_heads/n_kv_heads <= 8 (DEX_E_INVAL from
 * dex_create otherwise).                                                   */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  float rope_theta, rms_eps, residual_scale;
  int32_t weight_dtype;                 /* dex_dtype */
  const void *embed;                    /* device [vocab][d] */
  const float *final_norm;              /* device [d] */
  const void *lm_head;                  /* device [vocab][d] */
  const void *const *layers;            /* HOST array [n_layers * DEX_P_COUNT] of device pointers */
} dex_model;

/* "An explored-depth set" plus execution limits. */
typedef struct {
  const int32_t *explored;              /* host [n_explored], strictly increasing in [1, L], last == L */
  int32_t n_explored;                   /* N, 1 .. DEX_MAX_EXPLORED */
  int32_t width_cap;                    /* lattice rows per round per sequence; 0 = uncapped
                                           (the paper's binary lattice, needs 2^(N-1) rows) */
  int32_t decs;                         /* 1: DECS masked argmax (Algorithm 2, greedy); 0: plain argmax */
  int32_t batch;                        /* independent sequences, 1 .. DEX_MAX_BATCH */
  int32_t max_context;                  /* prompt length + generated tokens, per sequence */
  void *hip_stream;                     /* hipStream_t or NULL */
  int32_t stage_streams;                /* streams (lanes) a round's stages are spread
                                           over: the stages of one round read and write
                                           disjoint state, so they may run concurrently.
                                           0: the library default; 1: everything on
                                           hip_stream */
  float temperature;                    /* 0: greedy decoding.  > 0: Algorithm 2's sampling
                                           mode, every node decodes argmax(l / temperature
                                           + G) with G the Gumbel row of (sample_seed,
                                           sequence, position of the node's input token)
                                           (see dex_debug_gumbel below) */
  uint64_t sample_seed;
  int32_t adapter_dim;                  /* 0: no adapters.  Else m, the hidden width of the
                                           inducing adapters (Section 3.4 and its appendix):
                                           a node at a non-final explored depth k decodes
                                           h + dh_k(h), dh = alpha (W2 silu(W1 RMSNorm(h; g)
                                           + b1) + b2); the final depth is never adapted */
  const void *const *adapters;          /* [n_explored - 1][6] device pointers per non-final
                                           depth: g float[d], W1 [m][d], b1 float[m],
                                           W2 [d][m], b2 float[d], alpha float[1]; matrices in
                                           weight_dtype.  Borrowed: read at create (the
                                           library keeps repacked copies and alpha) */
  int32_t stage_grouping;               /* 0 (default) or 1: each lane takes a contiguous run
                                           of the round's stages and runs them in step, each
                                           kernel launched once per layer step for every
                                           stage of the run that has that step; -1: each
                                           stage's layers launched on their own, the stages
                                           dealt round-robin over the lanes.  The results
                                           are the same bits either way. */
} dex_config;

/* What one dex_step did (all host memory).  Rows are listed stage-major,
 * then by sequence, then in the lattice's priority order.                  */
typedef struct {
  int32_t n_rows;                       /* lattice nodes evaluated this round, all sequences */
  int32_t rows_per_stage[DEX_MAX_EXPLORED];
  int32_t layers_streamed;              /* layers of the stages that had >= 1 row */
  int32_t row_layers;                   /* sum over rows of the layers each row ran */
  int32_t q[DEX_MAX_BATCH];             /* FSM state (anchor's completed stages) at round start */
  int32_t kstar[DEX_MAX_BATCH];         /* shallowest matching depth index if committed, else -1 */
  int32_t row_seq[DEX_MAX_ROWS];
  int32_t row_slot[DEX_MAX_ROWS];       /* canonical slot index within its sequence's lattice */
  int32_t row_stage[DEX_MAX_ROWS];
  int32_t row_pos[DEX_MAX_ROWS];        /* absolute position of the row's input token */
  int32_t row_token[DEX_MAX_ROWS];      /* decoded candidate (DECS argmax) of the row */
  int64_t rounds_total;                 /* dex_step calls so far */
  double attn_bytes;                    /* algorithmic bytes of the round's attention: keys and
                                           values of every position up to each row group's
                                           deepest row, at every layer it ran, plus the
                                           queries read and the outputs written */
} dex_step_info;

/* Validate the model and X, derive the stages, allocate caches and scratch.
 * Errors: DEX_E_INVAL (dims, X not strictly increasing / not ending at L,
 * rows per round above DEX_MAX_ROWS), DEX_E_NOMEM, DEX_E_HIP.              */
dex_status dex_create(const dex_model *model, const dex_config *config, dex_ctx **out);

/* Algorithm 1's init.  prompts: host [batch][prompt_len] token ids in
 * [0, vocab).  Writes first_tokens[batch] (host): y_0 per sequence.  May be
 * called again to restart decoding with new prompts.
 * Errors: DEX_E_INVAL (ids, lengths), DEX_E_CAPACITY (prompt_len >= max_context). */
dex_status dex_prefill(dex_ctx *ctx, const int32_t *prompts, int32_t prompt_len, int32_t *first_tokens);

/* One round for every sequence.  committed (host [batch]): the token a
 * sequence committed this round, or -1.  info may be NULL.  A sequence whose
 * committed length reached max_context takes no further part.
 * Errors: DEX_E_STATE (no prefill yet / poisoned), DEX_E_CAPACITY (every
 * sequence is full, or the lattice outgrew its slot capacity), DEX_E_HIP.   */
dex_status dex_step(dex_ctx *ctx, int32_t *committed, dex_step_info *info);

/* Frees every library-owned allocation.  NULL-safe. */
void dex_destroy(dex_ctx *ctx);

const char *dex_last_error(const dex_ctx *ctx);

/* ---------------------------------------------------------------------------
 * Inspection taps for tests and the benchmark.
 * ------------------------------------------------------------------------- */

/* The work items the planner picks for one lattice state (host only: no
 * context and no GPU are needed).  Algorithm 1's expansion with the
 * eligibility of the one-explorer-per-device pipeline (a non-anchor slot
 * advances only when every ancestor has completed more stages) and the
 * width-cap priority (not in the paper, which names branch pruning as future
 * work): the anchor's advance first, then the width_cap - 1 other items of
 * lowest (hypothesis cost, path length, path), where a path is the string of
 * depth steps (a slot's stage k to k+1) and position steps (a slot's stage f
 * to the stage-0 node of the slot forked there) from the anchor's stage-0
 * node to the item's node, compared with the depth step first, and the
 * hypothesis cost is the sum of f + 1 over the fork stages f on it.
 *   slots      host [n_slots][4 + n_explored] int32, canonical order, slot 0
 *              the anchor: parent (-1 for slot 0, else an earlier slot),
 *              fork stage (< the parent's c, <= n_explored - 2; at most one
 *              child per (parent, stage)), c (completed stages), absolute
 *              position, then the candidates u[0..c-1] (the rest ignored)
 *   out        host [capacity][3] int32: kind (0 advance, 1 fork), slot,
 *              fork stage (-1 for advance), in priority order; *n_out = count
 * width_cap 0 = uncapped.  Malformed slots or too small a capacity:
 * DEX_E_INVAL (*n_out still receives the count in the latter case).        */
dex_status dex_debug_plan(int32_t n_explored, int32_t width_cap, int32_t decs, int32_t max_context,
                          const int32_t *slots, int32_t n_slots, int32_t *out, int32_t capacity, int32_t *n_out);

/* While enabled, every dex_step writes the float32 exit logits (before the
 * DECS mask) of each round row r to device_buf + r * vocab.  capacity_rows
 * must be >= the rows a round can have.  device_buf NULL disables.          */
dex_status dex_debug_set_logits_tap(dex_ctx *ctx, float *device_buf, int32_t capacity_rows);

/* Slot table of sequence `seq` in canonical order, each slot written as
 * stride = 5 + N int32: x, pos, parent (-1 for the anchor), fork stage, c,
 * then u[0..N-1] (-1 where not computed).  *n_slots receives the count.     */
dex_status dex_debug_lattice(dex_ctx *ctx, int32_t seq, int32_t *out, int32_t capacity_slots, int32_t *n_slots);

/* The last collapse of sequence `seq`: old canonical indices of the retained
 * slots (in order), whether the new anchor is fresh, and the committed
 * position the old anchor's keys/values went to.                            */
dex_status dex_debug_last_collapse(dex_ctx *ctx, int32_t seq, int32_t *map, int32_t capacity,
                                   int32_t *n_map, int32_t *fresh, int32_t *committed_pos);

/* Key/value cache layout: element (layer l, seq s, kv head g, entry e, dim i)
 * is at base + (((l * batch + s) * n_kv_heads + g) * entries + e) * head_dim + i
 * with entries returned in *entries.  Entry p < max_context is committed
 * position p; lattice slot j of seq s lives at entry lattice_entry(s, j)
 * (see dex_debug_slot_entry).                                                */
dex_status dex_debug_kv_layout(dex_ctx *ctx, void **k_base, void **v_base, int64_t *entries);
dex_status dex_debug_slot_entry(dex_ctx *ctx, int32_t seq, int32_t slot, int32_t *entry);

/* Kernel timing: while enabled, hipEvents bracket every launch of the layer
 * kernels on the context's stream.  dex_debug_kernel_times fills, for each
 * kernel class c < n (0 qkv, 1 attention, 2 attention combine, 3 o-proj,
 * 4 gate/up, 5 down, 6 lm-head, 7 other), the summed milliseconds and the
 * launch count since the last reset, and the algorithmic bytes moved by those
 * launches (weights + activations + keys/values they read or write).          */
dex_status dex_debug_set_kernel_timing(dex_ctx *ctx, int32_t enable);
dex_status dex_debug_kernel_times(dex_ctx *ctx, int32_t n, double *ms, int64_t *launches, double *bytes);

/* Round phases: while enabled, dex_step records events on the decode stream
 * at its boundaries.  dex_debug_round_times fills, summed over the rounds
 * since the last enable (*rounds of them), in milliseconds:
 *   ms[0] row-table upload           ms[1] stage sweep (all lanes joined)
 *   ms[2] exit head, verify/commit    ms[3] result copy to the host
 *   ms[4] host commit handling and the collapse gather (from the copy's
 *         end to the collapse's end; one round fewer than *rounds)
 *   ms[5] the gap before a round: from the previous round's last device
 *         work to this round's upload (return to the caller, the caller's
 *         own work, the next call's planning; one round fewer)
 *   ms[6] host planning (dex_step entry to the upload, host clock)
 * n <= 7 entries are written.                                               */
dex_status dex_debug_set_round_timing(dex_ctx *ctx, int32_t enable);
dex_status dex_debug_round_times(dex_ctx *ctx, int32_t n, double *ms, int64_t *rounds);

/* Mean duration of one decode-step GEMM class (3 o-proj, 4 gate/up, 5 down,
 * 6 lm-head) at M rows: `reps` back-to-back launches on the context's stream
 * between two hipEvents, cycling through the layers' weights so that no
 * launch re-reads a matrix another launch just streamed.  Uses the context's
 * scratch buffers (the decode state is untouched).  *bytes_per_launch is the
 * algorithmic traffic of one launch (weights plus activations).            */
dex_status dex_debug_time_kernel(dex_ctx *ctx, int32_t cls, int32_t M, int32_t reps, double *avg_us,
                                 double *bytes_per_launch);

/* Stand-alone GEMM y[M][N] = x[M][K] * W[N][K]^T (float32 out).  M in
 * [1, 64] runs the skinny matrix-core kernel the decode step uses (tests of
 * batch invariance); M > 64 (bf16 only, N a multiple of 16) runs the M-tiled
 * kernel of the prompt prefill.  dtype: dex_dtype of W and x; K a multiple of
 * 8 (bf16) or 4 (fp32).  Device pointers.                                   */
dex_status dex_debug_gemm(int32_t dtype, const void *W, int32_t N, int32_t K, const void *x, int32_t M,
                          float *y, void *hip_stream);

/* Stand-alone decode attention (K4, the branch-masked attention of one
 * layer) with its split combine, launched exactly as a step launches them
 * for one stage.  Row r (sequence row_seq[r], absolute position row_pos[r],
 * committed length row_nc[r]) attends with every query head h to the
 * logical keys 0..row_pos[r] of kv head h / (n_heads / n_kv_heads): cache
 * entries 0..row_nc[r]-1 of its sequence, then entry chain[chain_off[r] + t]
 * for position row_nc[r] + t (its ancestor slots and its own slot), with
 * scale 1/sqrt(head_dim) and softmax over those keys.  Consecutive rows of
 * one sequence with equal row_nc form a row group as in a step.
 *   dtype      dex_dtype of the caches and of out (bf16: matrix-core kernel
 *              for head_dim 64 and 128)
 *   head_dim   32, 64 or 128; n_heads a multiple of n_kv_heads, at most 8
 *              query heads per kv head
 *   k_cache, v_cache  device [batch][n_kv_heads][kv_entries][head_dim]
 *   q          device float [n_rows][n_heads * head_dim] (RoPE applied)
 *   out        device [n_rows][n_heads * head_dim] of dtype
 *   row_*, chain_off, chain   host arrays (n_rows entries; chain_len)
 * Requires 0 <= row_seq < batch, 0 <= row_nc <= row_pos + 1 <= kv_entries,
 * at most 64 chain positions per row (row_pos - row_nc < 64), chain entries
 * in [0, kv_entries) and chain_off[r] + row_pos[r] - row_nc[r] < chain_len;
 * anything else returns DEX_E_INVAL before any launch.  Allocates and frees
 * its own tables and split partials; synchronises hip_stream.            */
dex_status dex_debug_attention(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                               int32_t batch, int32_t kv_entries, const void *k_cache, const void *v_cache,
                               const float *q, int32_t n_rows, const int32_t *row_seq, const int32_t *row_pos,
                               const int32_t *row_nc, const int32_t *chain_off, const int32_t *chain,
                               int32_t chain_len, void *out, void *hip_stream);

/* dex_debug_attention for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): same arguments, same kernels and the same output bits, but
 * the row tables and split partials live in a fixed array of 64 MiB that
 * the library holds on every GPU it runs on until the process ends (the
 * first call on a device resolves that device's copy; the call runs on the
 * current device, which must own hip_stream).  No hipMalloc, hipFree or
 * other allocating routine is called.  Limits: n_rows <= DEX_MAX_ROWS,
 * chain_len <= 16384, and n_rows * n_heads * (max row_pos / 64 + 1) *
 * (head_dim + 2) * 4 bytes of split partials <= 63.75 MiB (at head_dim 128
 * and 32 heads: 8 rows up to 32128 keys each); beyond them
 * the call returns DEX_E_CAPACITY before any device work, with the reason
 * in dex_last_error(NULL).  Every call on one GPU shares that GPU's array:
 * calls that overlap on one GPU (other threads, other streams) race and must
 * be serialised by the caller.  Nothing in the array needs to start at zero
 * (every partial the combine reads is written by the same call).
 * Synchronises hip_stream.                                                  */
dex_status dex_debug_attention_noalloc(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                                       int32_t batch, int32_t kv_entries, const void *k_cache,
                                       const void *v_cache, const float *q, int32_t n_rows,
                                       const int32_t *row_seq, const int32_t *row_pos, const int32_t *row_nc,
                                       const int32_t *chain_off, const int32_t *chain, int32_t chain_len,
                                       void *out, void *hip_stream);

/* The Gumbel source of sampling mode (Algorithm 2 draws one Gumbel row per
 * sampling slot; here the row of a slot is a function of (seed, sequence,
 * position of the slot's input token), so plain autoregressive sampling at
 * the same position draws the same row and the committed tokens equal AR
 * sampling's).  With the SplitMix64 finaliser mix64 and gamma =
 * 0x9E3779B97F4A7C15 (Steele, Lea and Flood, OOPSLA 2014), all mod 2^64:
 *   key = mix64(seed ^ mix64(seq * 2^32 + pos)),
 *   z_v = mix64(key + (v + 1) * gamma),
 *   u_v = ((z_v >> 41) + 1/2) / 2^23      (exact in binary32),
 *   G_v = -ln(-ln u_v)                    (binary32 here).
 * dex_debug_gumbel writes G_0..G_{V-1} of one row to device memory `out`
 * (float32) on `hip_stream`, for tests of the generator.                    */
dex_status dex_debug_gumbel(uint64_t seed, int32_t seq, int32_t pos, int32_t V, float *out, void *hip_stream);

/* Plain device copy of `bytes` (multiple of 16) used to calibrate hardware
 * traffic counters against a kernel of known size.                          */
dex_status dex_debug_copy(void *dst, const void *src, int64_t bytes, void *hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* DEX_H */
