// The decode attention work item on the matrix cores (bf16 caches, head_dim
// 64 or 128) as a device function of one wave, and the wave-level helpers
// the attention kernels share.
#pragma once

#include "dex_kernels.h"

namespace dex {

typedef __attribute__((ext_vector_type(8))) __bf16 pf_bf16x8;
typedef __attribute__((ext_vector_type(4))) float pf_f32x4;

__device__ __forceinline__ uint16_t pf_f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
// Two floats rounded to bf16 (nearest even, as pf_f2bf) and packed, low first.
typedef __attribute__((ext_vector_type(2))) __bf16 pf_bf16x2;
typedef __attribute__((ext_vector_type(2))) float pf_f32x2;
__device__ __forceinline__ uint32_t pf_pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((pf_f32x2{lo, hi}), pf_bf16x2));
}
// Max and sum over a wave: xor butterfly, so every lane ends with the same bits.
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

// LDS written by some lanes of a wave and read by others: the wave's LDS
// operations complete in order once counted out; no other wave takes part.
__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_wave_barrier();
}

// Decode attention on the matrix cores (bf16 caches, head_dim 64 or 128).
//
// Same partials as attn_kernel -- (o, max, sum) per (row, query head, split
// of 64 logical keys) -- with the two products on v_mfma_f32_16x16x32_bf16:
//   S^T = K Q^T  the split's four 16-key tiles against the (row, query
//                head) pairs as 16 columns, q rounded to bf16: each lane
//                then holds 16 keys of one pair;
//   O^T = V^T P^T  P = exp(S - max) rounded to bf16 straight from those
//                accumulators (the B operand's k-slots are ordered as the
//                keys the lane holds), V staged row-major in LDS and read
//                back in the same key order through the transpose read
//                (tr_frag) as the A operand; each lane then holds four
//                consecutive dimensions of its own pair per 16-dimension
//                tile and writes them, rounded to bf16, with one 8-byte
//                store.  (The same
//                registers as an O = P V product with the operands swapped:
//                the product's bits are the same, and the split record needs
//                8 vector stores per lane instead of 32 scalar ones.)
// Keys are loaded in fragment order (16 keys x 64 bytes per instruction),
// values as whole key rows (four per instruction): value loads of one key
// row per lane touch 64 cache lines per instruction and held the split's
// loads to 4.4 TB/s.  A split whose keys are consecutive committed entries
// visible to every pair (the common case at long context) takes straight
// address arithmetic and no mask.
// Each output element of an MFMA depends only on its own pair's row and its
// key (or dimension) column, and the softmax statistics reduce over the
// split's keys in a fixed order (the lane's 16 keys in sequence, then the
// four quarter-waves as an xor butterfly), so a pair gets the same bits
// whichever pairs share its tile.
//
// Work items, one wave each, per kv head:
//   chain items  (row, first or second split holding the row's lattice
//                chain positions [nc, pos]): the row alone, its keys read
//                from the committed cache below nc and from its chain
//                entries from nc on.  A chain spans at most N + 1 <= 33
//                positions, so two splits.  Dispatched first.
//   group items  (row group, split): every row of the group that reaches
//                the split and has no chain positions in it, committed
//                keys only.  A split below the group's committed length
//                (every split but the last at long context) takes all of
//                the group's rows and needs none of their positions, so
//                its keys are requested right after the group's table
//                entries instead of after a further round trip for the
//                rows' positions.
// An MFMA 16x16x32 bf16 operand fragment from a key-major LDS tile with two
// transpose reads (ds_read_b64_tr_b16).  Within each quarter-wave, lane j
// receives element i from the address of lane 4 i + j / 4 at offset j % 4;
// so if the lane (quarter q, 4 i + g) addresses row R(q, i) at column 4 g of
// a tile, lane (column c, quarter q) gets rows R(q, 0..3) of column c as its
// first four k-slots, and the second read's rows as the next four.  Key rows
// of V are padded to hd + 16 elements, so four consecutive rows start 8 banks
// apart and a quarter-wave's read is conflict-free.
typedef __attribute__((ext_vector_type(4))) short tr_i16x4;
__device__ __forceinline__ pf_bf16x8 tr_frag(const uint16_t *lo, const uint16_t *hi) {
  const tr_i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) tr_i16x4 *)lo);
  const tr_i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) tr_i16x4 *)hi);
  const uint2 ua = __builtin_bit_cast(uint2, a), ub = __builtin_bit_cast(uint2, b);
  return __builtin_bit_cast(pf_bf16x8, make_uint4(ua.x, ua.y, ub.x, ub.y));
}

template <int HD>
__device__ void attn_mfma_item(const AttnArgs &a, int item, int kvh, uint16_t (*vr)[HD + 16], int *prow, int *ppos) {
  constexpr int KS = HD / 32;                 // k-steps of S over head dims
  constexpr int DT = HD / 16;                 // 16-dim tiles of O
  constexpr int NKT = ATT_SPLIT / 16;         // 16-key tiles per split
  constexpr int V4 = HD / 8;                  // 16-byte chunks per key row
  // vr: the split's value rows; prow / ppos: rows (relative to r0) of the
  // pass and their positions
  const int lane = threadIdx.x & 63, r16 = lane & 15, grp = lane >> 4;
  const int G = a.n_heads / a.n_kv_heads;
  const int n_chain_items = 2 * a.n_rows;
  int r0, seq, split, n_pass;
  int c_nc = 0, c_pos = -1, c_coff = 0;       // chain item: its row
  int tn;                                     // group item: committed keys of the split
  bool full = false;                          // every key of the split is seen by every pair
  const bool chain_item = item < n_chain_items;
  if (chain_item) {
    r0 = item >> 1;
    c_pos = a.row_pos[r0];
    c_nc = a.row_nc[r0];
    c_coff = a.row_chain_off[r0];
    seq = a.row_seq[r0];
    if (c_pos < c_nc) return;                   // no chain keys
    split = c_nc / ATT_SPLIT + (item & 1);
    if (split * ATT_SPLIT > c_pos) return;
    n_pass = 1;
    if (lane == 0) { prow[0] = 0; ppos[0] = c_pos; }
    tn = 0;
  } else {
    const int gi = (item - n_chain_items) / a.n_splits;
    split = a.n_splits - 1 - (item - n_chain_items) % a.n_splits;
    r0 = a.grp_row0[gi];
    seq = a.grp_seq[gi];
    const int nr = a.grp_nrows[gi];
    const int s0 = split * ATT_SPLIT, s1 = s0 + ATT_SPLIT - 1;
    if (a.grp_nc != nullptr && s1 < a.grp_nc[gi]) {
      // a split wholly inside the group's committed prefix: every row of the
      // group reaches past it and has no chain position in it, so all of
      // them take every key -- the decisions below, read off the group alone
      n_pass = nr;
      if (lane < nr) { prow[lane] = lane; ppos[lane] = INT_MAX; }
      tn = ATT_SPLIT;
      full = true;
    } else {
      // lane rr holds row rr of the group (at most 64 rows)
      const bool lr = lane < nr;
      const int mypos = lr ? a.row_pos[r0 + lane] : -1;
      const int mync = lr ? a.row_nc[r0 + lane] : 0;
      int maxpos = mypos, ncmax = mync;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        maxpos = max(maxpos, __shfl_xor(maxpos, o, 64));
        ncmax = max(ncmax, __shfl_xor(ncmax, o, 64));
      }
      if (s0 > maxpos) return;
      // a row whose chain positions fall in this split gets it from its chain
      // item; the pass takes the group's other rows that reach the split
      const bool chain_here = lr && max(mync, s0) <= min(mypos, s1);
      const bool in_pass = mypos >= s0 && !chain_here;
      const unsigned long long reach = __ballot(in_pass);
      if (reach == 0ull) return;
      n_pass = __popcll(reach);
      if (in_pass) {
        const int k = __popcll(reach & ((1ull << lane) - 1ull));
        prow[k] = lane;
        ppos[k] = mypos;
      }
      tn = max(0, min(ATT_SPLIT, ncmax - s0));
      int minpos = in_pass ? mypos : INT_MAX;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) minpos = min(minpos, __shfl_xor(minpos, o, 64));
      full = tn == ATT_SPLIT && s1 <= minpos;
    }
  }
  wave_lds_sync();
  const int s0 = split * ATT_SPLIT;
  const uint16_t *kbase = (const uint16_t *)a.kc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;
  const uint16_t *vbase = (const uint16_t *)a.vc + ((size_t)seq * a.n_kv_heads + kvh) * a.kv_entries * HD;
  // cache entry of key position s0 + j: committed below nc, then the chain;
  // -1 past what any row of the item attends to
  auto entry = [&](int j) -> int {
    const int kp = s0 + j;
    if (chain_item) return kp < c_nc ? kp : (kp <= c_pos ? a.chain[c_coff + (kp - c_nc)] : -1);
    return j < tn ? kp : -1;
  };

  // K as B fragments in registers: kf[nt][st] = key s0 + 16 nt + r16, dims
  // 32 st + 8 grp .. +8
  // V: whole key rows per load instruction (lane: row c * RPI + lane / V4,
  // 16-byte chunk lane % V4), stored row-major; the P.V operands are read
  // back with the LDS transpose read (see tr_frag)
  constexpr int RPI = 64 / V4;                // key rows per load instruction
  const int vrow = lane / V4, vch = lane % V4;
  uint4 kf[NKT][KS], vv[V4];
  if (full) {                                 // consecutive cache entries s0 ..
    const uint16_t *kb = kbase + (size_t)s0 * HD, *vb = vbase + (size_t)s0 * HD;
#pragma unroll
    for (int nt = 0; nt < NKT; ++nt)
#pragma unroll
      for (int st = 0; st < KS; ++st)
        kf[nt][st] = *(const uint4 *)(kb + (nt * 16 + r16) * HD + st * 32 + grp * 8);
#pragma unroll
    for (int c = 0; c < V4; ++c) vv[c] = *(const uint4 *)(vb + (c * RPI + vrow) * HD + vch * 8);
  } else {
#pragma unroll
    for (int nt = 0; nt < NKT; ++nt) {
      const int e = entry(nt * 16 + r16);
#pragma unroll
      for (int st = 0; st < KS; ++st)
        kf[nt][st] = e >= 0 ? *(const uint4 *)(kbase + (size_t)e * HD + st * 32 + grp * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < V4; ++c) {
      const int e = entry(c * RPI + vrow);
      vv[c] = e >= 0 ? *(const uint4 *)(vbase + (size_t)e * HD + vch * 8) : make_uint4(0, 0, 0, 0);
    }
  }
#pragma unroll
  for (int c = 0; c < V4; ++c) *(uint4 *)&vr[c * RPI + vrow][vch * 8] = vv[c];
  wave_lds_sync();

  // this lane as a transpose-read source: quarter tq, key ti within it,
  // four-element column group tg
  const int tq = lane >> 4, ti = (lane & 15) >> 2, tg = lane & 3;
  const int P = n_pass * G;
  for (int mt = 0; mt * 16 < P; ++mt) {
    // Q^T fragments: pair mt*16 + r16, dims 32 st + 8 grp .. +8 (bf16)
    const int pa = mt * 16 + r16;
    const bool pok = pa < P;
    const int row = r0 + (pok ? prow[pa / G] : 0);
    const float *qsrc = a.q + (size_t)row * a.ldq + (kvh * G + (pok ? pa % G : 0)) * HD + grp * 8;
    pf_bf16x8 qf[KS];
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
      if (pok) {
        x0 = *(const float4 *)(qsrc + st * 32);
        x1 = *(const float4 *)(qsrc + st * 32 + 4);
      }
      const uint4 u = make_uint4(pf_pack_bf16(x0.x, x0.y), pf_pack_bf16(x0.z, x0.w),
                                 pf_pack_bf16(x1.x, x1.y), pf_pack_bf16(x1.z, x1.w));
      qf[st] = __builtin_bit_cast(pf_bf16x8, u);
    }
    // S^T = K Q^T: lane holds key 16 nt + 4 grp + i against its own pair pa
    pf_f32x4 sc[NKT];
#pragma unroll
    for (int nt = 0; nt < NKT; ++nt) sc[nt] = pf_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KS; ++st)
#pragma unroll
      for (int nt = 0; nt < NKT; ++nt)
        sc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(pf_bf16x8, kf[nt][st]), qf[st], sc[nt], 0, 0, 0);
    // softmax over the split for pair pa: 16 keys in this lane (nt, i order),
    // then the lanes pa + 16, pa + 32 (xor butterfly over the four quarters)
    const int pos = pok ? ppos[pa / G] : -1;
    float mx = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < NKT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = sc[nt][i] * a.scale;
        if (!full && s0 + nt * 16 + grp * 4 + i > pos) v = -INFINITY;
        sc[nt][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = 0.f;
#pragma unroll
    for (int nt = 0; nt < NKT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float e = (mx == -INFINITY) ? 0.f : expf(sc[nt][i] - mx);
        sum += e;
        sc[nt][i] = e;
      }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    // O^T = V^T P^T: the transpose reads of V (the A operand) and the P
    // fragment (B) are the registers an O = P V product would use, swapped,
    // so each lane holds four consecutive dimensions of its own pair pa
    pf_f32x4 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = pf_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < ATT_SPLIT / 32; ++st) {
      // P^T (32 keys x pairs): k-slot e of lane (pair r16, grp) is key
      // 32 st + 4 grp + e (e < 4) or 32 st + 16 + 4 grp + e - 4, exactly the
      // S^T values this lane holds; V^T's k-slots follow the same key order
      const pf_bf16x8 pfr = __builtin_bit_cast(
          pf_bf16x8, make_uint4(pf_pack_bf16(sc[2 * st][0], sc[2 * st][1]), pf_pack_bf16(sc[2 * st][2], sc[2 * st][3]),
                                pf_pack_bf16(sc[2 * st + 1][0], sc[2 * st + 1][1]),
                                pf_pack_bf16(sc[2 * st + 1][2], sc[2 * st + 1][3])));
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            tr_frag(&vr[32 * st + 4 * tq + ti][16 * dt + 4 * tg], &vr[32 * st + 16 + 4 * tq + ti][16 * dt + 4 * tg]),
            pfr, o[dt], 0, 0, 0);
    }
    // pair pa's record: O[pa][16 dt + 4 grp .. + 3] rounded to bf16, one
    // 8-byte store per tile, and its statistics from the first quarter
    if (pok) {
      const size_t rec = ((size_t)(r0 + prow[pa / G]) * a.n_heads + kvh * G + pa % G) * a.jmax + split;
      uint16_t *dst = (uint16_t *)a.part + rec * HD + 4 * grp;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *(uint2 *)(dst + 16 * dt) = make_uint2(pf_pack_bf16(o[dt][0], o[dt][1]), pf_pack_bf16(o[dt][2], o[dt][3]));
      if (grp == 0) *(float2 *)(a.stat + 2 * rec) = make_float2(mx, sum);
    }
  }
}


}  // namespace dex
